// Plan kernel: the kept decode positions of one step (Algorithm 1, section 4),
// and the state-reset kernel.
//
// One wave per (request, KV head).  The skip list is stored as offsets
// d = t - j that never change (every list entry and t advance by one per
// step), so "shift skip_idx by +1" is free and the kept set at step t is
//   { t - d : 0 <= d <= min(t, N_r - 1), d not in the first n entries }
// with n = clamp(t - N_att + 1, 0, N_r - N_att) entries appended at earlier
// steps.  d <= N_r - 1 is the live window [t - N_r + 1, t]: in phase 3 row
// t - N_r is evicted in the same step, so it is never attended.
#include "device.h"
#include "internal.h"

namespace dsa {
namespace {

__global__ __launch_bounds__(kBlock) void plan_kernel(PlanArgs a) {
  extern __shared__ uint32_t bitmap_all[];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int pair = blockIdx.x * kWaves + wave;
  const bool live = pair < a.pairs;
  uint32_t* bm = bitmap_all + wave * a.words;

  // Every load of the wave is issued before any of them is used: the
  // decode position, the stored count and the first kPre*64 stored offsets
  // (entries past the count are ignored).
  const bool diag = a.mode == DSA_MODE_DIAGONAL;
  const uint16_t* off = a.st_off + static_cast<size_t>(pair) * a.state_cap;
  int t = live ? a.pos[pair / a.Hkv] : -1;
  const int cnt = (live && diag) ? a.st_count[pair] : 0;
  constexpr int kPre = 8;
  int dv[kPre];
#pragma unroll
  for (int i = 0; i < kPre; ++i) {
    const int e = lane + 64 * i;
    dv[i] = (live && diag && e < a.state_cap) ? off[e] : 0;
  }
  int flags = 0, nuse = 0;
  if (live) {
    if (t < 0) {
      flags = DSA_FLAG_INACTIVE;
    } else if (t >= a.Ldec) {
      t = a.Ldec - 1;
      flags = DSA_FLAG_POS_CLAMPED;
    }
  }
  if (live && diag && t >= 0) {
    const int nvalid = min(max(t - a.Natt + 1, 0), a.state_cap);
    if (cnt < nvalid) flags |= DSA_FLAG_STATE_BEHIND;
    nuse = min(max(cnt, 0), nvalid);
  }
  if (diag) {
    for (int w = lane; w < a.words; w += 64) bm[w] = 0u;
  }
  __syncthreads();
  if (diag && live && t >= 0) {
    bool bad = false;
#pragma unroll
    for (int i = 0; i < kPre; ++i) {
      const int e = lane + 64 * i;
      if (e < nuse) {
        const int d = dv[i];
        if (d <= a.Nr - 2) atomicOr(&bm[d >> 5], 1u << (d & 31)); else bad = true;
      }
    }
    for (int e = lane + 64 * kPre; e < nuse; e += 64) {
      const int d = off[e];
      if (d <= a.Nr - 2) atomicOr(&bm[d >> 5], 1u << (d & 31)); else bad = true;
    }
    if (__ballot(bad)) flags |= DSA_FLAG_BAD_OFFSET;
  }
  __syncthreads();
  if (!live) return;

  if (t < 0) {
    if (lane == 0) {
      a.count[pair] = 0;
      a.flags[pair] = flags;
    }
    return;
  }
  if (!diag) {
    if (lane == 0) {
      a.count[pair] = t + 1;
      a.flags[pair] = flags;
    }
    return;
  }

  // Ascending positions p = t - d for d = dmax .. 0, compacted by ballot.
  const int dmax = min(t, a.Nr - 1);
  int32_t* out = a.idx + static_cast<size_t>(pair) * a.plan_cap;
  const uint64_t below = (uint64_t(1) << lane) - 1;
  int n = 0;
  for (int p0 = t - dmax; p0 <= t; p0 += 64) {
    const int p = p0 + lane;
    bool kept = false;
    if (p <= t) {
      const int d = t - p;
      kept = ((bm[d >> 5] >> (d & 31)) & 1u) == 0u;
    }
    const uint64_t mask = __ballot(kept);
    const int slot = n + __popcll(mask & below);
    if (kept && slot < a.plan_cap) out[slot] = p;
    n += __popcll(mask);
  }
  if (lane == 0) {
    if (!(flags & (DSA_FLAG_STATE_BEHIND | DSA_FLAG_BAD_OFFSET)) && n != min(t + 1, a.Natt))
      flags |= DSA_FLAG_COUNT;
    a.count[pair] = min(n, a.plan_cap);
    a.flags[pair] = flags;
  }
}

__global__ __launch_bounds__(256) void reset_kernel(ResetArgs a) {
  const int pair = blockIdx.x * 256 + threadIdx.x;
  if (pair >= a.pairs) return;
  if (a.mask && a.mask[pair / a.Hkv] == 0) return;
  a.st_count[pair] = 0;
  a.st_flags[pair] = 0;
}

}  // namespace

hipError_t launch_plan(const Derived& d, const PlanArgs& a, hipStream_t st) {
  const int pairs = d.B * d.Hkv;
  const int grid = (pairs + kWaves - 1) / kWaves;
  const size_t lds = d.mode == DSA_MODE_DIAGONAL ? sizeof(uint32_t) * kWaves * a.words : 0;
  plan_kernel<<<grid, kBlock, lds, st>>>(a);
  return hipGetLastError();
}

hipError_t launch_reset(const Derived& d, const ResetArgs& a, hipStream_t st) {
  const int grid = (a.pairs + 255) / 256;
  reset_kernel<<<grid, 256, 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace dsa

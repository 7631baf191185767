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
//
// With S sinks (section 5.1) positions 0 .. S-1 are kept first and the rule
// above applies to the later positions with t - S in place of t and
// N_att - S in place of N_att: offsets 0 .. min(t - S, W - 1), the first
// clamp(t - N_att + 1, 0, cap) stored offsets skipped.  Window mode is the
// same with W = N_att - S and no stored offsets.
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
  const bool sparse = a.mode != DSA_MODE_DENSE;
  const bool stated = a.state_cap > 0;  // diagonal mode with a skip list
  const uint16_t* off = a.st_off + static_cast<size_t>(pair) * a.state_cap;
  int t = live ? a.pos[pair / a.Hkv] : -1;
  const int cnt = (live && stated) ? a.st_count[pair] : 0;
  constexpr int kPre = 8;
  int dv[kPre];
#pragma unroll
  for (int i = 0; i < kPre; ++i) {
    const int e = lane + 64 * i;
    dv[i] = (live && stated && e < a.state_cap) ? off[e] : 0;
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
  if (live && stated && t >= 0) {
    const int nvalid = min(max(t - a.Natt + 1, 0), a.state_cap);
    if (cnt < nvalid) flags |= DSA_FLAG_STATE_BEHIND;
    nuse = min(max(cnt, 0), nvalid);
  }
  for (int w = lane; w < a.words; w += 64) bm[w] = 0u;
  __syncthreads();
  if (nuse > 0) {
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
  if (!sparse) {
    if (lane == 0) {
      a.count[pair] = t + 1;
      a.flags[pair] = flags;
    }
    return;
  }

  // The sinks, then ascending positions p = t - d for d = dmax .. 0,
  // compacted by ballot (dmax < 0 while t < S: no window yet).
  const int sk = min(a.Ns, t + 1);
  const int dmax = min(t - a.Ns, a.Nr - 1);
  int32_t* out = a.idx + static_cast<size_t>(pair) * a.plan_cap;
  for (int r = lane; r < sk; r += 64) out[r] = r;
  const uint64_t below = (uint64_t(1) << lane) - 1;
  int n = sk;
  for (int p0 = t - dmax; p0 <= t; p0 += 64) {
    const int p = p0 + lane;
    bool kept = false;
    if (p <= t) {
      const int d = t - p;
      kept = nuse == 0 || ((bm[d >> 5] >> (d & 31)) & 1u) == 0u;
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
  a.st_kc[2 * pair] = 0;
  a.st_kc[2 * pair + 1] = 0;
}

}  // namespace

hipError_t launch_plan(const Derived& d, const PlanArgs& a, hipStream_t st) {
  const int pairs = d.B * d.Hkv;
  const int grid = (pairs + kWaves - 1) / kWaves;
  const size_t lds = sizeof(uint32_t) * kWaves * a.words;
  plan_kernel<<<grid, kBlock, lds, st>>>(a);
  return hipGetLastError();
}

hipError_t launch_reset(const Derived& /*d*/, const ResetArgs& a, hipStream_t st) {
  const int grid = (a.pairs + 255) / 256;
  reset_kernel<<<grid, 256, 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace dsa

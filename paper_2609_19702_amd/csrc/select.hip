// Select kernel: the phase-2 argmin of Algorithm 1 (section 4).
//
// At a step t with N_att - 1 <= t <= N_r - 2 every KV head appends one skip
// entry: the kept window key with the lowest softmax weight.  The window
// softmax is taken over the kept decode keys only (the prompt is not part of
// K[idx]).  With several query heads per KV head, the weights of the group
// are summed; with one, the argmin is taken on the logits themselves, which
// the softmax orders identically.  Ties go to the first (oldest) key.  The
// entry is stored as the offset t - idx[j*] at list slot k = t - N_att + 1,
// so running the same step twice rewrites the same slot.
//
// With S sinks the steps that select are N_att - 1 <= t <= N_r + S - 2 (the
// phase-2 range of the positions after the sinks), the sinks are the first
// S kept positions and never candidates, and k = t - N_att + 1 still holds.
#include "device.h"
#include "internal.h"

namespace dsa {
namespace {

template <int G>
__global__ __launch_bounds__(kBlock) void select_kernel(SelectArgs a) {
  const int lane = threadIdx.x & 63;
  const int pair = blockIdx.x * kWaves + (threadIdx.x >> 6);
  if (pair >= a.pairs) return;
  const int b = pair / a.Hkv;
  const int kvh = pair % a.Hkv;
  int t = a.pos[b];
  const int cnt = a.st_count[pair];
  const int n = min(max(a.count[pair], 0), a.plan_cap);
  if (t < 0) return;
  t = min(t, a.Ldec - 1);
  if (t < a.Natt - 1 || t > a.Nr + a.Ns - 2) return;
  const int k = t - (a.Natt - 1);
  if (k >= a.state_cap) return;
  if (cnt < k) {
    if (lane == 0) a.st_flags[pair] |= DSA_FLAG_STATE_BEHIND;
    return;
  }
  const int nw = n - a.Ns;  // kept window keys after the sinks
  if (nw <= 0) return;
  const float* wl = a.wlog + (static_cast<size_t>(b) * a.Hq + kvh * G) * a.plan_cap + a.Ns;
  const int plan_cap = a.plan_cap;
  int jbest = window_argmin<G>(lane, nw, [&](int g, int j) { return wl[g * plan_cap + j]; });
  if (jbest < 0 || jbest >= nw) jbest = 0;  // only for NaN logits
  const int32_t* kept_pos = a.idx + static_cast<size_t>(pair) * a.plan_cap + a.Ns;
  if (lane == 0) {
    const int d = min(max(t - kept_pos[jbest], 0), a.Nr - 2);
    a.st_off[static_cast<size_t>(pair) * a.state_cap + k] = static_cast<uint16_t>(d);
    a.st_count[pair] = k + 1;
  }
  if (a.kept_on && nw == a.kept_cap) {
    const int sl = (k + 1) & 1;
    write_kept_list(lane, nw, jbest, t, a.Natt - a.Ns + k, [&](int r) { return kept_pos[r]; },
                    a.st_kept + (static_cast<size_t>(pair) * 2 + sl) * a.kept_stride,
                    a.st_kc + 2 * pair + sl, k + 1);
  }
}

}  // namespace

hipError_t launch_select(const Derived& d, const SelectArgs& a, hipStream_t st) {
  const int grid = (a.pairs + kWaves - 1) / kWaves;
  switch (d.G) {
    case 1: select_kernel<1><<<grid, kBlock, 0, st>>>(a); break;
    case 2: select_kernel<2><<<grid, kBlock, 0, st>>>(a); break;
    case 4: select_kernel<4><<<grid, kBlock, 0, st>>>(a); break;
    default: select_kernel<8><<<grid, kBlock, 0, st>>>(a); break;
  }
  return hipGetLastError();
}

}  // namespace dsa

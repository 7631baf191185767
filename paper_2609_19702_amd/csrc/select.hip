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
#include "device.h"
#include "internal.h"

namespace dsa {
namespace {

// (value, index) minimum with ties to the smaller index.
__device__ __forceinline__ void argmin_merge(float& v, int& j, float v2, int j2) {
  if (v2 < v || (v2 == v && j2 < j)) {
    v = v2;
    j = j2;
  }
}

__device__ __forceinline__ void wave_argmin(float& v, int& j) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    const float v2 = __shfl_xor(v, m, 64);
    const int j2 = __shfl_xor(j, m, 64);
    argmin_merge(v, j, v2, j2);
  }
}

template <int G>
__global__ __launch_bounds__(kBlock) void select_kernel(SelectArgs a) {
  const int lane = threadIdx.x & 63;
  const int pair = blockIdx.x * kWaves + (threadIdx.x >> 6);
  if (pair >= a.pairs) return;
  const int b = pair / a.Hkv;
  const int kvh = pair % a.Hkv;
  int t = a.pos[b];
  if (t < 0) return;
  t = min(t, a.Ldec - 1);
  if (t < a.Natt - 1 || t > a.Nr - 2) return;
  const int k = t - (a.Natt - 1);
  if (k >= a.state_cap) return;
  const int cnt = a.st_count[pair];
  if (cnt < k) {
    if (lane == 0) a.st_flags[pair] |= DSA_FLAG_STATE_BEHIND;
    return;
  }
  const int n = min(max(a.count[pair], 0), a.plan_cap);
  if (n == 0) return;
  const float* wl = a.wlog + (static_cast<size_t>(b) * a.Hq + kvh * G) * a.plan_cap;

  float best = __builtin_inff();
  int jbest = 0x7fffffff;
  if constexpr (G == 1) {
    for (int j = lane; j < n; j += 64) argmin_merge(best, jbest, wl[j], j);
  } else {
    // sigma_j = sum_g exp(s_gj - max_g) / sum_j' exp(s_gj' - max_g)
    float mx[G], inv[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float* w = wl + static_cast<size_t>(g) * a.plan_cap;
      float m = -__builtin_inff();
      for (int j = lane; j < n; j += 64) m = fmaxf(m, w[j]);
      m = wave_max(m);
      float s = 0.f;
      for (int j = lane; j < n; j += 64) s += __expf(w[j] - m);
      s = wave_sum(s);
      mx[g] = m;
      inv[g] = 1.f / s;
    }
    for (int j = lane; j < n; j += 64) {
      float sigma = 0.f;
#pragma unroll
      for (int g = 0; g < G; ++g)
        sigma += __expf(wl[static_cast<size_t>(g) * a.plan_cap + j] - mx[g]) * inv[g];
      argmin_merge(best, jbest, sigma, j);
    }
  }
  wave_argmin(best, jbest);
  if (lane == 0) {
    if (jbest < 0 || jbest >= n) jbest = 0;  // only for NaN logits
    const int pos = a.idx[static_cast<size_t>(pair) * a.plan_cap + jbest];
    const int d = min(max(t - pos, 0), a.Nr - 2);
    a.st_off[static_cast<size_t>(pair) * a.state_cap + k] = static_cast<uint16_t>(d);
    a.st_count[pair] = k + 1;
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

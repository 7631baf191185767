// Device helpers for gfx950 (CDNA4, 64-lane wavefronts).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace dsa {

// bf16 -> fp32 is exact: the bf16 bits are the high half of the fp32 bits.
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ void unpack8(const uint4& r, float (&f)[8]) {
  f[0] = bf16_lo(r.x);
  f[1] = bf16_hi(r.x);
  f[2] = bf16_lo(r.y);
  f[3] = bf16_hi(r.y);
  f[4] = bf16_lo(r.z);
  f[5] = bf16_hi(r.z);
  f[6] = bf16_lo(r.w);
  f[7] = bf16_hi(r.w);
}

// 16-byte global load with the non-temporal hint: K/V rows are streamed once
// per step, so they should not push the small per-step buffers (queries,
// selection state, plans) out of the caches.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 load_stream16(const void* p) {
  const u32x4 x = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return make_uint4(x.x, x.y, x.z, x.w);
}

// DPP lane permutations inside a 16-lane row.
constexpr int kDppQuadSwap1 = 0xB1;   // quad_perm [1,0,3,2]: lane ^ 1
constexpr int kDppQuadSwap2 = 0x4E;   // quad_perm [2,3,0,1]: lane ^ 2
constexpr int kDppRowMirror = 0x140;  // lane i <- lane 15 - i
constexpr int kDppHalfMirror = 0x141; // lane i <- lane 7 - i within each 8-lane half
constexpr int kDppRowRor8 = 0x128;    // lane i <- lane (i + 8) mod 16: lane ^ 8

template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}

// Sum over aligned groups of N lanes (N = 4, 8 or 16); every lane of a
// group receives the group's sum.  Pure DPP: no LDS traffic.
template <int N>
__device__ __forceinline__ float group_sum(float x) {
  static_assert(N == 4 || N == 8 || N == 16, "group of 4, 8 or 16 lanes");
  x += dpp<kDppQuadSwap1>(x);
  x += dpp<kDppQuadSwap2>(x);
  if constexpr (N >= 8) x += dpp<kDppHalfMirror>(x);
  if constexpr (N == 16) x += dpp<kDppRowMirror>(x);
  return x;
}

// ds_swizzle in bit mode: lane i reads lane i ^ 4 within each 32-lane half
// (and mask 0x1f, or mask 0, xor mask 4).
constexpr int kSwizzleXor4 = 0x1F | (4 << 10);

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// One step of a butterfly across lanes l and l ^ OFF (OFF = 4, 8, 16 or 32)
// without a trip through LDS memory: ds_swizzle for 4, a DPP row rotate for
// 8, the gfx950 lane swaps (v_permlane16_swap / v_permlane32_swap) for 16
// and 32.  Gives the pair as (first, second) with first the value of the
// lane whose bit OFF is clear, so every lane of that half sees (own,
// partner).
template <int OFF>
__device__ __forceinline__ void xor_pair(float x, float& first, float& second) {
  static_assert(OFF == 4 || OFF == 8 || OFF == 16 || OFF == 32,
                "butterfly step of 4, 8, 16 or 32 lanes");
  if constexpr (OFF == 4) {
    first = x;
    second = __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(x), kSwizzleXor4));
  } else if constexpr (OFF == 8) {
    first = x;
    second = dpp<kDppRowRor8>(x);
  } else {
    const uint32_t u = __float_as_uint(x);
    const auto r = OFF == 16 ? __builtin_amdgcn_permlane16_swap(u, u, false, false)
                             : __builtin_amdgcn_permlane32_swap(u, u, false, false);
    first = __uint_as_float(r[0]);
    second = __uint_as_float(r[1]);
  }
}

__device__ __forceinline__ float shfl_xor(float x, int mask) { return __shfl_xor(x, mask, 64); }

template <int CTRL>
__device__ __forceinline__ int dpp_i(int x) {
  return __builtin_amdgcn_update_dpp(0, x, CTRL, 0xF, 0xF, false);
}

// Reductions over the 64 lanes of a wave without the LDS crossbar: two quad
// permutations, the 8-lane half mirror and the 16-lane mirror (DPP) combine
// ever larger aligned groups, then the 16- and 32-lane swaps.  The operation
// must be commutative; every lane ends with the same value.
template <typename Op>
__device__ __forceinline__ float wave_allreduce(float x, Op op) {
  x = op(x, dpp<kDppQuadSwap1>(x));
  x = op(x, dpp<kDppQuadSwap2>(x));
  x = op(x, dpp<kDppHalfMirror>(x));
  x = op(x, dpp<kDppRowMirror>(x));
  float a, b;
  xor_pair<16>(x, a, b);
  x = op(a, b);
  xor_pair<32>(x, a, b);
  return op(a, b);
}

template <typename Op>
__device__ __forceinline__ int wave_allreduce(int x, Op op) {
  x = op(x, dpp_i<kDppQuadSwap1>(x));
  x = op(x, dpp_i<kDppQuadSwap2>(x));
  x = op(x, dpp_i<kDppHalfMirror>(x));
  x = op(x, dpp_i<kDppRowMirror>(x));
  float a, b;
  xor_pair<16>(__int_as_float(x), a, b);
  x = op(__float_as_int(a), __float_as_int(b));
  xor_pair<32>(__int_as_float(x), a, b);
  return op(__float_as_int(a), __float_as_int(b));
}

__device__ __forceinline__ float wave_max(float x) {
  return wave_allreduce(x, [](float a, float b) { return fmaxf(a, b); });
}

__device__ __forceinline__ float wave_sum(float x) {
  return wave_allreduce(x, [](float a, float b) { return a + b; });
}

}  // namespace dsa

namespace dsa {

// (value, index) minimum with ties to the smaller index.
__device__ __forceinline__ void argmin_merge(float& v, int& j, float v2, int j2) {
  if (v2 < v || (v2 == v && j2 < j)) {
    v = v2;
    j = j2;
  }
}

// Phase-2 selection score argmin of one KV head over its n kept window keys
// (section 4, Algorithm 1): logit(g, j) is sm_scale * q_g . k_j of query head
// g of the group for window key j.  Group size 1 takes the argmin of the
// logits (the softmax orders them identically); larger groups sum the
// group's window softmaxes.  Ties go to the smallest j (the oldest key).
// Called by a whole wave; every lane returns the same index (or a value
// outside [0, n) only if every score is NaN).
//
// Windows of up to kArgminRegs * 64 keys are read once, every load issued
// before the first use, and kept in registers for the max, sum and score
// passes; longer windows stream the logits once per pass.  Both forms add
// the same terms in the same order.
constexpr int kArgminRegs = 4;

template <int G, typename Logit>
__device__ __forceinline__ int window_argmin(int lane, int n, Logit logit) {
  float best = __builtin_inff();
  int jbest = 0x7fffffff;
  if (n <= 64 * kArgminRegs) {
    float v[G][kArgminRegs];
#pragma unroll
    for (int c = 0; c < kArgminRegs; ++c) {
      const int j = lane + 64 * c;
#pragma unroll
      for (int g = 0; g < G; ++g) v[g][c] = j < n ? logit(g, j) : -__builtin_inff();
    }
    if constexpr (G == 1) {
#pragma unroll
      for (int c = 0; c < kArgminRegs; ++c)
        if (lane + 64 * c < n) argmin_merge(best, jbest, v[0][c], lane + 64 * c);
    } else {
      float mx[G], inv[G];
#pragma unroll
      for (int g = 0; g < G; ++g) {
        float m = -__builtin_inff();
#pragma unroll
        for (int c = 0; c < kArgminRegs; ++c) m = fmaxf(m, v[g][c]);
        m = wave_max(m);
        float s = 0.f;
#pragma unroll
        for (int c = 0; c < kArgminRegs; ++c)
          if (lane + 64 * c < n) s += __expf(v[g][c] - m);
        s = wave_sum(s);
        mx[g] = m;
        inv[g] = 1.f / s;
      }
#pragma unroll
      for (int c = 0; c < kArgminRegs; ++c) {
        if (lane + 64 * c < n) {
          float sigma = 0.f;
#pragma unroll
          for (int g = 0; g < G; ++g) sigma += __expf(v[g][c] - mx[g]) * inv[g];
          argmin_merge(best, jbest, sigma, lane + 64 * c);
        }
      }
    }
  } else if constexpr (G == 1) {
    for (int j = lane; j < n; j += 64) argmin_merge(best, jbest, logit(0, j), j);
  } else {
    float mx[G], inv[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float m = -__builtin_inff();
      for (int j = lane; j < n; j += 64) m = fmaxf(m, logit(g, j));
      m = wave_max(m);
      float s = 0.f;
      for (int j = lane; j < n; j += 64) s += __expf(logit(g, j) - m);
      s = wave_sum(s);
      mx[g] = m;
      inv[g] = 1.f / s;
    }
    for (int j = lane; j < n; j += 64) {
      float sigma = 0.f;
#pragma unroll
      for (int g = 0; g < G; ++g) sigma += __expf(logit(g, j) - mx[g]) * inv[g];
      argmin_merge(best, jbest, sigma, j);
    }
  }
  // The smallest score over the wave, then the smallest index among the
  // lanes that hold it (each lane's jbest is its smallest index with its
  // best score, so ties still go to the smallest j).
  const float m = wave_allreduce(best, [](float a, float b) { return fminf(a, b); });
  const int jm = best == m ? jbest : 0x7fffffff;
  return wave_allreduce(jm, [](int a, int b) { return min(a, b); });
}

}  // namespace dsa

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

// The window's kept offsets for the step after a phase-2 selection (the
// list a selection state keeps, see dsa_state_layout): this step's kept
// window rank r (0 <= r < nwin, ascending positions pos(r)) has offset
// t - pos(r); the selected rank jsel leaves, and the offset the window gains
// at the next step, first_off, leads.  Largest offset first.  Lane 0 then
// tags the list with k_next + 1 (k_next: the skip entries stored after this
// selection).  Called by a whole wave.
template <typename Pos>
__device__ __forceinline__ void write_kept_list(int lane, int nwin, int jsel, int t, int first_off,
                                                Pos pos, uint16_t* kept, int32_t* tag,
                                                int k_next) {
  if (lane == 0) kept[0] = static_cast<uint16_t>(first_off);
  for (int r = lane; r < nwin; r += 64)
    if (r != jsel) kept[r < jsel ? r + 1 : r] = static_cast<uint16_t>(t - pos(r));
  if (lane == 0) *tag = k_next + 1;
}

// (value, index) minimum with ties to the smaller index.
__device__ __forceinline__ void argmin_merge(float& v, int& j, float v2, int j2) {
  if (v2 < v || (v2 == v && j2 < j)) {
    v = v2;
    j = j2;
  }
}

// The butterfly of wave_allreduce on N values at once.  Each value goes
// through the same steps in the same order as it would alone, so the result
// is bit for bit the same; the N exchanges of a step are independent, so a
// wave waits for one step's latency instead of N.
template <int N, typename Op>
__device__ __forceinline__ void wave_allreduce_n(float (&x)[N], Op op) {
#pragma unroll
  for (int i = 0; i < N; ++i) x[i] = op(x[i], dpp<kDppQuadSwap1>(x[i]));
#pragma unroll
  for (int i = 0; i < N; ++i) x[i] = op(x[i], dpp<kDppQuadSwap2>(x[i]));
#pragma unroll
  for (int i = 0; i < N; ++i) x[i] = op(x[i], dpp<kDppHalfMirror>(x[i]));
#pragma unroll
  for (int i = 0; i < N; ++i) x[i] = op(x[i], dpp<kDppRowMirror>(x[i]));
  float a[N], b[N];
#pragma unroll
  for (int i = 0; i < N; ++i) xor_pair<16>(x[i], a[i], b[i]);
#pragma unroll
  for (int i = 0; i < N; ++i) x[i] = op(a[i], b[i]);
#pragma unroll
  for (int i = 0; i < N; ++i) xor_pair<32>(x[i], a[i], b[i]);
#pragma unroll
  for (int i = 0; i < N; ++i) x[i] = op(a[i], b[i]);
}

// Unsigned integers in the order of the floats they come from (-0 counts as
// +0, as a float comparison does).  Not for NaN.
__device__ __forceinline__ uint32_t ordered_bits(float v) {
  const uint32_t u = __float_as_uint(v + 0.f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// The smallest 64-bit key over the wave (every lane receives it).
__device__ __forceinline__ uint64_t wave_min_u64(uint64_t x) {
  auto take = [](uint64_t a, uint32_t lo, uint32_t hi) {
    const uint64_t b = (static_cast<uint64_t>(hi) << 32) | lo;
    return b < a ? b : a;
  };
  x = take(x, dpp_i<kDppQuadSwap1>(static_cast<int>(x)), dpp_i<kDppQuadSwap1>(static_cast<int>(x >> 32)));
  x = take(x, dpp_i<kDppQuadSwap2>(static_cast<int>(x)), dpp_i<kDppQuadSwap2>(static_cast<int>(x >> 32)));
  x = take(x, dpp_i<kDppHalfMirror>(static_cast<int>(x)), dpp_i<kDppHalfMirror>(static_cast<int>(x >> 32)));
  x = take(x, dpp_i<kDppRowMirror>(static_cast<int>(x)), dpp_i<kDppRowMirror>(static_cast<int>(x >> 32)));
  float lo0, lo1, hi0, hi1;
  xor_pair<16>(__uint_as_float(static_cast<uint32_t>(x)), lo0, lo1);
  xor_pair<16>(__uint_as_float(static_cast<uint32_t>(x >> 32)), hi0, hi1);
  x = take((static_cast<uint64_t>(__float_as_uint(hi0)) << 32) | __float_as_uint(lo0),
           __float_as_uint(lo1), __float_as_uint(hi1));
  xor_pair<32>(__uint_as_float(static_cast<uint32_t>(x)), lo0, lo1);
  xor_pair<32>(__uint_as_float(static_cast<uint32_t>(x >> 32)), hi0, hi1);
  return take((static_cast<uint64_t>(__float_as_uint(hi0)) << 32) | __float_as_uint(lo0),
              __float_as_uint(lo1), __float_as_uint(hi1));
}

// The smallest (score, index) key over the wave: a lane's best is its
// smallest score (never NaN; +inf with index 0x7fffffff where it has no
// candidate) and jbest its smallest index with that score, so the key order
// gives the smallest score, then the smallest index.  Every lane returns it.
__device__ __forceinline__ int wave_argmin_key(float best, int jbest) {
  const uint64_t key = (static_cast<uint64_t>(ordered_bits(best)) << 32) |
                       static_cast<uint32_t>(jbest);
  return static_cast<int>(static_cast<uint32_t>(wave_min_u64(key)));
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
// the same terms in the same order.  The group's heads go through each
// pass side by side (their maxima and sums are reduced over the wave
// together), and the final (score, index) minimum is one reduction of
// packed keys.
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
      float mx[G], sm[G], inv[G];
#pragma unroll
      for (int g = 0; g < G; ++g) {
        mx[g] = -__builtin_inff();
#pragma unroll
        for (int c = 0; c < kArgminRegs; ++c) mx[g] = fmaxf(mx[g], v[g][c]);
      }
      wave_allreduce_n<G>(mx, [](float a, float b) { return fmaxf(a, b); });
      float e[G][kArgminRegs];  // the exponentials, computed once for both passes
#pragma unroll
      for (int g = 0; g < G; ++g) {
        sm[g] = 0.f;
#pragma unroll
        for (int c = 0; c < kArgminRegs; ++c) {
          e[g][c] = __expf(v[g][c] - mx[g]);
          if (lane + 64 * c < n) sm[g] += e[g][c];
        }
      }
      wave_allreduce_n<G>(sm, [](float a, float b) { return a + b; });
#pragma unroll
      for (int g = 0; g < G; ++g) inv[g] = 1.f / sm[g];
#pragma unroll
      for (int c = 0; c < kArgminRegs; ++c) {
        if (lane + 64 * c < n) {
          float sigma = 0.f;
#pragma unroll
          for (int g = 0; g < G; ++g) sigma += e[g][c] * inv[g];
          argmin_merge(best, jbest, sigma, lane + 64 * c);
        }
      }
    }
  } else if constexpr (G == 1) {
    for (int j = lane; j < n; j += 64) argmin_merge(best, jbest, logit(0, j), j);
  } else {
    float mx[G], sm[G], inv[G];
#pragma unroll
    for (int g = 0; g < G; ++g) mx[g] = -__builtin_inff();
    for (int j = lane; j < n; j += 64)
#pragma unroll
      for (int g = 0; g < G; ++g) mx[g] = fmaxf(mx[g], logit(g, j));
    wave_allreduce_n<G>(mx, [](float a, float b) { return fmaxf(a, b); });
#pragma unroll
    for (int g = 0; g < G; ++g) sm[g] = 0.f;
    for (int j = lane; j < n; j += 64)
#pragma unroll
      for (int g = 0; g < G; ++g) sm[g] += __expf(logit(g, j) - mx[g]);
    wave_allreduce_n<G>(sm, [](float a, float b) { return a + b; });
#pragma unroll
    for (int g = 0; g < G; ++g) inv[g] = 1.f / sm[g];
    for (int j = lane; j < n; j += 64) {
      float sigma = 0.f;
#pragma unroll
      for (int g = 0; g < G; ++g) sigma += __expf(logit(g, j) - mx[g]) * inv[g];
      argmin_merge(best, jbest, sigma, j);
    }
  }
  return wave_argmin_key(best, jbest);
}

// The selection of window_argmin (G > 1) in two parts, so the heads of a
// group can be taken by different waves of a workgroup.
//
// head_terms: one head's window softmax, in place: row[j] (the logit of
// window key j, 0 <= j < n) becomes exp(row[j] - max) / sum.  The maximum,
// the sum and the terms are the values window_argmin computes for the head
// (same operations, same order).  Windows of up to kArgminRegs * 64 keys are
// read into registers at once (every LDS read issued before the first use);
// longer ones are streamed.  Called by a whole wave.
__device__ __forceinline__ void head_terms(int lane, int n, float* row) {
  float mx[1] = {-__builtin_inff()};
  float sm[1] = {0.f};
  if (n <= 64 * kArgminRegs) {
    float v[kArgminRegs], e[kArgminRegs];
#pragma unroll
    for (int c = 0; c < kArgminRegs; ++c) {
      const float x = row[min(lane + 64 * c, n - 1)];
      v[c] = lane + 64 * c < n ? x : -__builtin_inff();
    }
#pragma unroll
    for (int c = 0; c < kArgminRegs; ++c) mx[0] = fmaxf(mx[0], v[c]);
    wave_allreduce_n<1>(mx, [](float a, float b) { return fmaxf(a, b); });
#pragma unroll
    for (int c = 0; c < kArgminRegs; ++c) {
      e[c] = __expf(v[c] - mx[0]);
      if (lane + 64 * c < n) sm[0] += e[c];
    }
    wave_allreduce_n<1>(sm, [](float a, float b) { return a + b; });
    const float inv = 1.f / sm[0];
#pragma unroll
    for (int c = 0; c < kArgminRegs; ++c)
      if (lane + 64 * c < n) row[lane + 64 * c] = e[c] * inv;
    return;
  }
  for (int j = lane; j < n; j += 64) mx[0] = fmaxf(mx[0], row[j]);
  wave_allreduce_n<1>(mx, [](float a, float b) { return fmaxf(a, b); });
  for (int j = lane; j < n; j += 64) sm[0] += __expf(row[j] - mx[0]);
  wave_allreduce_n<1>(sm, [](float a, float b) { return a + b; });
  const float inv = 1.f / sm[0];
  for (int j = lane; j < n; j += 64) row[j] = __expf(row[j] - mx[0]) * inv;
}

// terms_argmin: the argmin of sigma_j = sum over the group's heads g (in
// order) of term(g, j), the terms head_terms left; the same index
// window_argmin returns.  term(g, j) must be readable for every j < n.
// Called by a whole wave.
template <int G, typename Term>
__device__ __forceinline__ int terms_argmin(int lane, int n, Term term) {
  float best = __builtin_inff();
  int jbest = 0x7fffffff;
  if (n <= 64 * kArgminRegs) {
    float t[kArgminRegs][G];
#pragma unroll
    for (int c = 0; c < kArgminRegs; ++c)
#pragma unroll
      for (int g = 0; g < G; ++g) t[c][g] = term(g, min(lane + 64 * c, n - 1));
#pragma unroll
    for (int c = 0; c < kArgminRegs; ++c) {
      float sigma = 0.f;
#pragma unroll
      for (int g = 0; g < G; ++g) sigma += t[c][g];
      if (lane + 64 * c < n) argmin_merge(best, jbest, sigma, lane + 64 * c);
    }
  } else {
    for (int j = lane; j < n; j += 64) {
      float sigma = 0.f;
#pragma unroll
      for (int g = 0; g < G; ++g) sigma += term(g, j);
      argmin_merge(best, jbest, sigma, j);
    }
  }
  return wave_argmin_key(best, jbest);
}

}  // namespace dsa

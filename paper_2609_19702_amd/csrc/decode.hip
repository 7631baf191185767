// Split-K single-query decode attention over the prompt KV plus the kept (or,
// in dense mode, all) decode KV, and the cross-split log-sum-exp combine.
//
// Attn(Q_t, K_p + K[idx], V_p + V[idx]) of Algorithm 1 (section 4) for one
// (request, KV head, split) per workgroup.  The keys of a (request, KV head)
// are numbered r = 0 .. n-1: the L_p prompt rows, then the kept decode rows in
// plan order (dense mode: decode rows 0 .. t).  Split s covers keys
// [s*C, min(n, (s+1)*C)).
//
// Data path (HBM-bound: each bf16 K/V element is read once and used for one
// multiply-add per query head of the group):
//   - a lane loads 16 bytes (8 bf16) of a row, so a 64-lane wave loads
//     512/d rows per instruction with 128-bit coalesced accesses (one row =
//     d/8 consecutive lanes = one contiguous 128/256-byte segment);
//   - each wave keeps U row blocks of K and V in flight before using them;
//   - q.k partial sums are reduced inside the row's lane group with DPP row
//     permutations (no LDS);
//   - softmax runs online in fp32 (base-2 exponent with the scale folded
//     in), one running (max, sum, acc[8]) per lane and query head;
//   - lane groups, then the 4 waves (through LDS), are merged by log-sum-exp
//     at the end; one split writes the final output directly, several splits
//     write fp32 partials (acc[d], max, sum) that the combine kernel merges.
#include "device.h"
#include "internal.h"

namespace dsa {
namespace {

struct RowRange {
  int n;     // keys of this (request, KV head); 0 for an unused slot
  int t;     // decode position after clamping (or -1)
};

__device__ __forceinline__ RowRange row_range(const DecodeArgs& a, int b, int pair) {
  RowRange r;
  int t = a.pos[b];
  if (t < 0) {
    r.n = 0;
    r.t = -1;
    return r;
  }
  t = min(t, a.Ldec - 1);
  const int nwin = a.mode == DSA_MODE_DENSE ? t + 1 : min(max(a.count[pair], 0), a.plan_cap);
  r.n = a.Lp + nwin;
  r.t = t;
  return r;
}

template <int D, int G, int U>
__global__ __launch_bounds__(kBlock) void decode_kernel(DecodeArgs a) {
  constexpr int LPR = D / 8;       // lanes per row
  constexpr int RPI = 64 / LPR;    // rows per load instruction
  constexpr int RPB = RPI * U;     // rows per wave block
  __shared__ float red[kWaves][G][D + 2];

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int rg = lane / LPR;       // row group within the wave
  const int c = lane % LPR;        // 8-element column chunk
  const int s = blockIdx.x % a.S;
  const int pair = blockIdx.x / a.S;
  const int kvh = pair % a.Hkv;
  const int b = pair / a.Hkv;

  const RowRange rr = row_range(a, b, pair);
  const int n = rr.n;
  const int r0 = s * a.C;
  if (s > 0 && r0 >= n) return;
  const int r1 = min(n, r0 + a.C);
  const int nsplit = (n + a.C - 1) / a.C;

  const int64_t base = (a.row_base ? a.row_base[b] : static_cast<int64_t>(b) * a.sb) +
                       static_cast<int64_t>(kvh) * a.sh + c * 8;
  const uint16_t* kb = a.k + base;
  const uint16_t* vb = a.v + base;
  const int32_t* idx = a.idx + static_cast<size_t>(pair) * a.plan_cap;
  const bool dense = a.mode == DSA_MODE_DENSE;

  float qf[G][8];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const uint4 qr = *reinterpret_cast<const uint4*>(
        a.q + (static_cast<size_t>(b) * a.Hq + kvh * G + g) * D + c * 8);
    unpack8(qr, qf[g]);
  }
  float m[G], l[G], acc[G][8];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m[g] = kNegBig;
    l[g] = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[g][e] = 0.f;
  }

  for (int blk = r0 + wave * RPB; blk < r1; blk += kWaves * RPB) {
    int crow[U];
    bool ok[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int r = blk + u * RPI + rg;
      ok[u] = r < r1;
      int cr = r;
      if (ok[u] && !dense && r >= a.Lp) cr = a.Lp + min(max(idx[r - a.Lp], 0), rr.t);
      crow[u] = ok[u] ? cr : 0;
    }
    uint4 kr[U], vr[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      kr[u] = make_uint4(0, 0, 0, 0);
      if (ok[u]) kr[u] = *reinterpret_cast<const uint4*>(kb + crow[u] * a.sr);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      vr[u] = make_uint4(0, 0, 0, 0);
      if (ok[u]) vr[u] = *reinterpret_cast<const uint4*>(vb + crow[u] * a.sr);
    }

    float sc[U][G];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float kf[8];
      unpack8(kr[u], kf);
#pragma unroll
      for (int g = 0; g < G; ++g) {
        float x = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) x = fmaf(qf[g][e], kf[e], x);
        sc[u][g] = group_sum<LPR>(x);
      }
    }
    if (a.wlog) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int r = blk + u * RPI + rg;
        if (ok[u] && c == 0 && r >= a.Lp) {
#pragma unroll
          for (int g = 0; g < G; ++g)
            a.wlog[(static_cast<size_t>(b) * a.Hq + kvh * G + g) * a.plan_cap + (r - a.Lp)] =
                sc[u][g] * a.scale;
        }
      }
    }
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float mx = kNegBig;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        sc[u][g] *= a.scale_log2;
        if (ok[u]) mx = fmaxf(mx, sc[u][g]);
      }
      const float mnew = fmaxf(m[g], mx);
      const float alpha = fast_exp2(m[g] - mnew);
      m[g] = mnew;
      l[g] *= alpha;
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[g][e] *= alpha;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float vf[8];
      unpack8(vr[u], vf);
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float p = ok[u] ? fast_exp2(sc[u][g] - m[g]) : 0.f;
        l[g] += p;
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[g][e] = fmaf(p, vf[e], acc[g][e]);
      }
    }
  }

  // Merge the row groups of the wave (lanes c, c + LPR, c + 2*LPR, ...).
#pragma unroll
  for (int off = LPR; off < 64; off <<= 1) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float m2 = shfl_xor(m[g], off);
      const float l2 = shfl_xor(l[g], off);
      const float mn = fmaxf(m[g], m2);
      const float a1 = fast_exp2(m[g] - mn);
      const float a2 = fast_exp2(m2 - mn);
      l[g] = l[g] * a1 + l2 * a2;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float x2 = shfl_xor(acc[g][e], off);
        acc[g][e] = acc[g][e] * a1 + x2 * a2;
      }
      m[g] = mn;
    }
  }
  if (rg == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
#pragma unroll
      for (int e = 0; e < 8; ++e) red[wave][g][c * 8 + e] = acc[g][e];
      if (c == 0) {
        red[wave][g][D] = m[g];
        red[wave][g][D + 1] = l[g];
      }
    }
  }
  __syncthreads();
  if (wave != 0) return;

  // Merge the 4 waves; lane j handles columns j and j + 64.
#pragma unroll
  for (int g = 0; g < G; ++g) {
    float M = kNegBig;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) M = fmaxf(M, red[w][g][D]);
    float L = 0.f, A0 = 0.f, A1 = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const float sw = fast_exp2(red[w][g][D] - M);
      L += red[w][g][D + 1] * sw;
      A0 += red[w][g][lane] * sw;
      if constexpr (D == 128) A1 += red[w][g][lane + 64] * sw;
    }
    const int h = kvh * G + g;
    if (nsplit <= 1) {
      const float inv = L > 0.f ? 1.f / L : 0.f;
      float* o = a.out + (static_cast<size_t>(b) * a.Hq + h) * D;
      o[lane] = A0 * inv;
      if constexpr (D == 128) o[lane + 64] = A1 * inv;
    } else {
      float* pp = a.part + ((static_cast<size_t>(pair) * a.S + s) * G + g) * (D + 2);
      pp[lane] = A0;
      if constexpr (D == 128) pp[lane + 64] = A1;
      if (lane == 0) {
        pp[D] = M;
        pp[D + 1] = L;
      }
    }
  }
}

// One wave per (request, query head): out = sum_s e^{m_s - M} acc_s /
// sum_s e^{m_s - M} l_s over the request's splits (base-2 exponents, as the
// partial maxima are kept in log2 units).
template <int D>
__global__ __launch_bounds__(kBlock) void combine_kernel(DecodeArgs a, int G) {
  const int lane = threadIdx.x & 63;
  const int bh = blockIdx.x * kWaves + (threadIdx.x >> 6);
  if (bh >= a.B * a.Hq) return;
  const int b = bh / a.Hq;
  const int h = bh % a.Hq;
  const int kvh = h / G;
  const int g = h % G;
  const int pair = b * a.Hkv + kvh;
  const RowRange rr = row_range(a, b, pair);
  const int nsplit = (rr.n + a.C - 1) / a.C;
  if (nsplit <= 1) return;
  const float* pp = a.part + (static_cast<size_t>(pair) * a.S * G + g) * (D + 2);
  const size_t sstride = static_cast<size_t>(G) * (D + 2);
  float M = kNegBig;
  for (int s = lane; s < nsplit; s += 64) M = fmaxf(M, pp[s * sstride + D]);
  M = wave_max(M);
  float L = 0.f;
  for (int s = lane; s < nsplit; s += 64) L += pp[s * sstride + D + 1] * fast_exp2(pp[s * sstride + D] - M);
  L = wave_sum(L);
  float A0 = 0.f, A1 = 0.f;
  for (int s = 0; s < nsplit; ++s) {
    const float sw = fast_exp2(pp[s * sstride + D] - M);
    A0 += pp[s * sstride + lane] * sw;
    if constexpr (D == 128) A1 += pp[s * sstride + lane + 64] * sw;
  }
  const float inv = L > 0.f ? 1.f / L : 0.f;
  float* o = a.out + static_cast<size_t>(bh) * D;
  o[lane] = A0 * inv;
  if constexpr (D == 128) o[lane + 64] = A1 * inv;
}

template <int D, int G>
hipError_t launch_dg(const Derived& d, const DecodeArgs& a, hipStream_t st) {
  const int grid = d.B * d.Hkv * d.S;
  if (d.U >= 4)
    decode_kernel<D, G, 4><<<grid, kBlock, 0, st>>>(a);
  else
    decode_kernel<D, G, 2><<<grid, kBlock, 0, st>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || d.S <= 1) return e;
  const int cgrid = (d.B * d.Hq + kWaves - 1) / kWaves;
  combine_kernel<D><<<cgrid, kBlock, 0, st>>>(a, G);
  return hipGetLastError();
}

template <int D>
hipError_t launch_d(const Derived& d, const DecodeArgs& a, hipStream_t st) {
  switch (d.G) {
    case 1: return launch_dg<D, 1>(d, a, st);
    case 2: return launch_dg<D, 2>(d, a, st);
    case 4: return launch_dg<D, 4>(d, a, st);
    default: return launch_dg<D, 8>(d, a, st);
  }
}

}  // namespace

hipError_t launch_decode(const Derived& d, const DecodeArgs& a, hipStream_t st) {
  return d.D == 64 ? launch_d<64>(d, a, st) : launch_d<128>(d, a, st);
}

}  // namespace dsa

// Split-K single-query decode attention over the prompt KV plus the kept (or,
// in dense mode, all) decode KV; the cross-split log-sum-exp combine; and the
// fused decode step that also builds the kept set and runs the phase-2
// selection.
//
// Attn(Q_t, K_p + K[idx], V_p + V[idx]) of Algorithm 1 (section 4) for one
// (request, KV head, split) per workgroup.  The keys of a (request, KV head)
// are numbered r = 0 .. n-1: the L_p prompt rows, then the kept decode rows in
// ascending position (dense mode: decode rows 0 .. t).  Split s covers keys
// [s*C, min(n, (s+1)*C)).
//
// Data path (HBM-bound: each K/V element is read once and used for one
// multiply-add per query head of the group):
//   - a lane loads 16 bytes of a row (8 bf16 or 16 fp8 elements), so a
//     64-lane wave loads 512/d (bf16) or 1024/d (fp8) rows per instruction
//     with 128-bit coalesced accesses (one row = consecutive lanes covering
//     one contiguous 64- to 256-byte segment);
//   - a wave works on tiles of U load instructions (at most 64 rows) and
//     issues every K and V load of a tile before using any of them; rows
//     past the end of the split read a valid row and get weight 0, so no
//     load sits behind a branch;
//   - tiles hold either prompt rows or kept decode rows, never both; the
//     kept positions of a window tile are held one per lane and handed to
//     the row groups with ds_bpermute, prompt tiles need none;
//   - K/V rows are loaded with the non-temporal hint (streamed once);
//   - with a ring layout a kept decode position j >= S (S sinks) is read
//     from slot S + (j - S) mod (ring - S) (the ring holds the sinks and the
//     live window; evicted rows are gone);
//   - a workgroup has as many waves (1..4) as its split has tiles, so no wave
//     sits idle holding registers;
//   - q.k partial sums are reduced inside the row's lane group with DPP row
//     permutations (no LDS);
//   - softmax runs online in fp32 (base-2 exponent with the scale folded
//     in), one running (max, sum, acc[8]) per lane and query head;
//   - lane groups, then the waves (through LDS), are merged by log-sum-exp at
//     the end; one split writes the final output directly, several splits
//     write fp32 partials (acc[d], max, sum) that a second kernel merges.
//
// The fused step (FUSED = true, diagonal mode) reads the selection state
// instead of a plan: each wave that owns kept decode rows rebuilds the skip
// set of its (request, KV head) as a bitmap in its own LDS slice and ranks the
// window positions with ballots, writing the plan as a by-product, before
// any wave of the workgroup starts loading K/V (the workgroup then streams
// all its rows together rather than the kept rows trailing); when one
// split covers the whole (request, KV head) the same workgroup then runs the
// phase-2 argmin on the window logits it computed and appends the skip entry.
// Every value it produces is bit-identical to dsa_plan -> dsa_decode_attention
// -> dsa_select.  The same path serves the sink variants of section 5.1: the
// S sinks are the first S kept ranks, the window rule applies to the later
// positions, and window mode (no stored offsets) skips the bitmap.
//
// This header holds the kernels as templates over the K/V element type
// (KvBf16, KvFp8); decode.hip and decode_fp8.hip each instantiate one.
#pragma once

#include <hip/hip_ext.h>

#include "device.h"
#include "internal.h"

namespace dsa {
namespace {

// K/V element types.  A lane always loads 16 consecutive bytes of a row (one
// 128-bit access): 8 bf16 elements or 16 fp8 elements (kEpl).  The tiles,
// row groups and reductions follow from the lanes per row, D / kEpl; only
// the widening to fp32 (or to the bf16 MFMA operand) differs.
struct KvBf16 {
  static constexpr int kBytes = 2;
  static constexpr int kEpl = 8;
  using Raw = uint4;
  static __device__ __forceinline__ Raw load(const uint8_t* p) { return load_stream16(p); }
  static __device__ __forceinline__ void widen(const Raw& r, float (&f)[8]) { unpack8(r, f); }
  // The bf16 MFMA operand of elements 8*half .. 8*half + 7 of a load.
  static __device__ __forceinline__ bf16x8 to_bf16(const Raw& r, int /*half*/) {
    return __builtin_bit_cast(bf16x8, r);
  }
};

struct KvFp8 {
  static constexpr int kBytes = 1;
  static constexpr int kEpl = 16;
  using Raw = uint4;
  static __device__ __forceinline__ Raw load(const uint8_t* p) { return load_stream16(p); }
  // v_cvt_pk_f32_fp8 widens two OCP E4M3 bytes (the low or the high half of
  // a word) to fp32 exactly.
  static __device__ __forceinline__ void widen_word(uint32_t w, float* f) {
    const auto lo = __builtin_amdgcn_cvt_pk_f32_fp8(static_cast<int>(w), false);
    const auto hi = __builtin_amdgcn_cvt_pk_f32_fp8(static_cast<int>(w), true);
    f[0] = lo[0];
    f[1] = lo[1];
    f[2] = hi[0];
    f[3] = hi[1];
  }
  static __device__ __forceinline__ void widen(const Raw& r, float (&f)[16]) {
    widen_word(r.x, f);
    widen_word(r.y, f + 4);
    widen_word(r.z, f + 8);
    widen_word(r.w, f + 12);
  }
  // Every E4M3 value is a bf16 value (4 significant bits, exponents
  // -9 .. 8), so keeping the high half of the fp32 bits is exact.
  static __device__ __forceinline__ bf16x8 to_bf16(const Raw& r, int half) {
    float f[8];
    widen_word(half ? r.z : r.x, f);
    widen_word(half ? r.w : r.y, f + 4);
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      w[i] = (__float_as_uint(f[2 * i]) >> 16) | (__float_as_uint(f[2 * i + 1]) & 0xffff0000u);
    return __builtin_bit_cast(bf16x8, make_uint4(w[0], w[1], w[2], w[3]));
  }
};

constexpr int kPre = 8;  // words per lane loaded ahead of the position (see PreRegs)

// Keys of the (request, KV head) and the clamped decode position.
struct RowRange {
  int n;      // keys; 0 for an unused slot
  int t;      // decode position after clamping, or -1
  int flags;  // DSA_FLAG_INACTIVE / DSA_FLAG_POS_CLAMPED
};

// From the raw decode position t and, for a plan-driven call, the plan's
// kept count.
template <bool FUSED>
__device__ __forceinline__ RowRange row_range_of(const DecodeArgs& a, int t, int plan_count) {
  RowRange r{0, -1, 0};
  if (t < 0) {
    r.flags = DSA_FLAG_INACTIVE;
    return r;
  }
  if (t >= a.Ldec) {
    t = a.Ldec - 1;
    r.flags = DSA_FLAG_POS_CLAMPED;
  }
  int nwin;
  if (a.mode == DSA_MODE_DENSE)
    nwin = t + 1;
  else if (FUSED)
    nwin = min(t + 1, a.Natt);  // the kept count of Algorithm 1 at step t
  else
    nwin = min(max(plan_count, 0), a.plan_cap);
  r.n = a.Lp + nwin;
  r.t = t;
  return r;
}

template <bool FUSED>
__device__ __forceinline__ RowRange row_range(const DecodeArgs& a, int b, int pair) {
  return row_range_of<FUSED>(a, a.pos[b],
                             (FUSED || a.mode == DSA_MODE_DENSE) ? 0 : a.count[pair]);
}

// Wave-private skip set of one (request, KV head) for the fused step: the
// bitmap of the first nuse stored offsets, plus the ranking cursor.
struct SkipSet {
  uint32_t* bm;
  int t, dmax;   // window offsets 0 .. dmax (dmax < 0: no window yet)
  int sk;        // sinks kept ahead of the window: min(S, t + 1)
  bool any;      // the bitmap holds at least one skipped offset
  int p0, rank;  // next candidate chunk and kept positions before it
  int flags;
};

__device__ __forceinline__ void fence_wave() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

// What a wave that may own window rows loads ahead of the decode position
// (kPre 16-bit values per lane), by the build:
//   without kept lists (KL false): the first kPre*64 stored skip offsets,
//     for the bitmap;
//   with them (KL true): the first 256 offsets of both kept lists (slot 0
//     for an even number of skip entries, slot 1 for an odd one; the step's
//     slot is known once the position arrives), kPre/2 values per lane and
//     slot.
// Branch-free, so the loads stay in flight until the ranking uses them and
// the waits before their first use count exactly these loads: entries past
// the data re-read entry 0, and a wave that needs none (use = false) reads
// a dummy address (the queries); the values are then unused.
struct PreRegs {
  uint32_t w[kPre];
};

template <bool KL>
__device__ __forceinline__ void load_pre(const DecodeArgs& a, int pair, int lane, bool use,
                                         PreRegs& pr) {
  constexpr int kl = KL ? 1 : 0;
  const int stride = (a.kept_cap + 1) & ~1;
  const int lim = use ? (kl ? a.kept_cap : a.state_cap) : 0;
  const uint16_t* kept = a.st_kept + static_cast<size_t>(pair) * 2 * stride;
  const uint16_t* off = a.st_off + static_cast<size_t>(pair) * a.state_cap;
  const uint16_t* base = lim > 0 ? (kl ? kept : off) : reinterpret_cast<const uint16_t*>(a.q);
#pragma unroll
  for (int i = 0; i < kPre; ++i) {
    const int e = lane + 64 * (i - kl * (i & (kPre / 2)));  // list mode: i mod kPre/2
    const int so = kl * (i / (kPre / 2)) * stride;          // list mode: the slot's start
    pr.w[i] = base[e < lim ? so + e : 0];
  }
}

// The skip bitmap from the first `cnt` stored offsets that the step at
// decode position t uses.  In the build without kept lists (KL false) the
// first kPre*64 of them are already in registers; in the other one (the
// step's kept list is missing) they are all read here.
template <bool KL>
__device__ void build_skip_set(const DecodeArgs& a, int pair, int lane, int t, int cnt,
                               uint32_t* bm, const PreRegs& pr, SkipSet& ss) {
  const uint16_t* off = a.st_off + static_cast<size_t>(pair) * a.state_cap;
  for (int w = lane; w < a.words; w += 64) bm[w] = 0u;
  const int nvalid = min(max(t - a.Natt + 1, 0), a.state_cap);
  int flags = cnt < nvalid ? DSA_FLAG_STATE_BEHIND : 0;
  const int nuse = min(max(cnt, 0), nvalid);
  fence_wave();
  bool bad = false;
  int e0 = 0;
  if constexpr (!KL) {
#pragma unroll
    for (int i = 0; i < kPre; ++i) {
      const int e = lane + 64 * i;
      if (e < nuse) {
        const int d = static_cast<int>(pr.w[i]);
        if (d <= a.Nr - 2) atomicOr(&bm[d >> 5], 1u << (d & 31)); else bad = true;
      }
    }
    e0 = 64 * kPre;
  }
  for (int e = lane + e0; e < nuse; e += 64) {
    const int d = off[e];
    if (d <= a.Nr - 2) atomicOr(&bm[d >> 5], 1u << (d & 31)); else bad = true;
  }
  if (__ballot(bad)) flags |= DSA_FLAG_BAD_OFFSET;
  fence_wave();
  ss.bm = bm;
  ss.t = t;
  ss.sk = min(a.Ns, t + 1);
  ss.dmax = min(t - a.Ns, a.Nr - 1);
  ss.any = nuse > 0;
  ss.p0 = t - ss.dmax;
  ss.rank = ss.sk;
  ss.flags = flags;
}

__device__ __forceinline__ bool is_kept(const SkipSet& ss, int p) {
  if (p > ss.t) return false;
  if (!ss.any) return true;
  const int d = ss.t - p;
  return ((ss.bm[d >> 5] >> (d & 31)) & 1u) == 0u;
}

// Kept window positions of ranks [lo, hi) (ascending position), written to
// kp[rank - kp_base] (LDS; the plan rows are written from there after the
// K/V loop, so no store waits behind the loads in the memory queue).  The
// cursor only moves forward, so the tiles of a wave (in increasing rank
// order) share one scan.  The scan reads
// the bitmap words of kRankBatch chunks of 64 positions at once, so the LDS
// latency is paid once per batch rather than once per chunk.
constexpr int kRankBatch = 4;

__device__ void rank_window(int lane, SkipSet& ss, int lo, int hi, int* kp, int kp_base) {
  const uint64_t below = (uint64_t(1) << lane) - 1;
  for (int r = lo + lane; r < min(hi, ss.sk); r += 64)  // sink rank r is position r
    kp[r - kp_base] = r;
  bool more = ss.p0 <= ss.t && ss.rank < hi;
  while (more) {
    bool kept[kRankBatch];
    uint64_t mask[kRankBatch];
#pragma unroll
    for (int i = 0; i < kRankBatch; ++i) kept[i] = is_kept(ss, ss.p0 + 64 * i + lane);
#pragma unroll
    for (int i = 0; i < kRankBatch; ++i) mask[i] = __ballot(kept[i]);
#pragma unroll
    for (int i = 0; i < kRankBatch && more; ++i) {
      const int p = ss.p0 + lane;
      const int rk = ss.rank + __popcll(mask[i] & below);
      if (kept[i] && rk >= lo && rk < hi) kp[rk - kp_base] = p;
      const int tot = ss.rank + __popcll(mask[i]);
      if (tot > hi) {  // the chunk reaches past this tile: keep it for the next one
        more = false;
      } else {
        ss.rank = tot;
        ss.p0 += 64;
        more = ss.p0 <= ss.t && ss.rank < hi;
      }
    }
  }
  fence_wave();
}

// Total kept positions of the window (for the DSA_FLAG_COUNT check).
__device__ int count_kept(const SkipSet& ss, int lane) {
  int n = ss.sk;
  for (int p0 = ss.t - ss.dmax; p0 <= ss.t; p0 += 64 * kRankBatch) {
    bool kept[kRankBatch];
#pragma unroll
    for (int i = 0; i < kRankBatch; ++i) kept[i] = is_kept(ss, p0 + 64 * i + lane);
#pragma unroll
    for (int i = 0; i < kRankBatch; ++i) n += __popcll(__ballot(kept[i]));
  }
  return n;
}

// One butterfly step of the log-sum-exp merge of per-lane partial results
// (running max m, sum l, weighted values acc) across lanes l and l ^ OFF.
// Every lane whose bit OFF is clear combines (own, partner) in that order.
template <int OFF, int G, int EPL>
__device__ __forceinline__ void merge_groups(float (&m)[G], float (&l)[G], float (&acc)[G][EPL]) {
#pragma unroll
  for (int g = 0; g < G; ++g) {
    float m1, m2, l1, l2;
    xor_pair<OFF>(m[g], m1, m2);
    xor_pair<OFF>(l[g], l1, l2);
    const float mn = fmaxf(m1, m2);
    const float a1 = fast_exp2(m1 - mn);
    const float a2 = fast_exp2(m2 - mn);
    l[g] = fmaf(l1, a1, l2 * a2);
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      float x1, x2;
      xor_pair<OFF>(acc[g][e], x1, x2);
      acc[g][e] = fmaf(x1, a1, x2 * a2);
    }
    m[g] = mn;
  }
}

// Round to the nearest bf16 (ties to even); finite inputs.
__device__ __forceinline__ uint32_t bf16_rne_bits(float x) {
  const uint32_t u = __float_as_uint(x);
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

// Rows of a wave's V tile in LDS are D + kVPad bf16 apart: 32 bytes past a
// multiple of 128, so the four rows one transposed read touches fall in
// distinct banks.
constexpr int kVPad = 16;

typedef short s16x4 __attribute__((ext_vector_type(4)));

// K and V of one 32-row tile of the grouped-head path, as loaded (the loads
// of two tiles can be in flight at once: mf_load issues, mf_compute waits).
template <class KV, int D>
struct MfRaw {
  static constexpr int EPL = KV::kEpl, KPL = EPL / 8, LPR = D / EPL, RPI = 64 / LPR;
  static constexpr int NK = D / 32, UV = kMfmaTile / RPI, NH = kMfmaTile / 16;
  typename KV::Raw k[NH][NK / KPL];
  typename KV::Raw v[UV];
};

// Rows [rs, re) of a tile; window tiles read row Lp + pos_l of lane i for
// row rs + i (pos_l: the kept position, or its ring slot).
template <class KV, int D>
__device__ __forceinline__ void mf_load(const DecodeArgs& a, int lane, int rs, int re,
                                        bool has_win, int pos_l, const uint8_t* kmf,
                                        const uint8_t* vb, MfRaw<KV, D>& raw) {
  using R = MfRaw<KV, D>;
  const int lr = lane & 15, rg = lane / R::LPR;
  // K load li of lane group lq holds elements 32*KPL*li + EPL*lq .. + EPL-1,
  // the A operands of k-steps KPL*li .. KPL*li + KPL-1 (the queries use the
  // same element order; q.k does not depend on it).
#pragma unroll
  for (int h = 0; h < R::NH; ++h) {
    const int r = rs + 16 * h + lr;
    const int wpos = has_win ? __shfl(pos_l, 16 * h + lr, 64) : 0;
    int cr = 0;  // rows past the tile end read row 0 and get weight 0
    if (r < re) cr = has_win ? a.Lp + wpos : r;
#pragma unroll
    for (int li = 0; li < R::NK / R::KPL; ++li)
      raw.k[h][li] = KV::load(kmf + cr * a.sr + 32 * R::KPL * KV::kBytes * li);
  }
#pragma unroll
  for (int u = 0; u < R::UV; ++u) {
    const int r = rs + u * R::RPI + rg;
    const int wpos = has_win ? __shfl(pos_l, u * R::RPI + rg, 64) : 0;
    int cr = 0;
    if (r < re) cr = has_win ? a.Lp + wpos : r;
    raw.v[u] = KV::load(vb + cr * a.sr);
  }
}

// One 32-row tile of the grouped-head path, both products on the matrix
// cores (v_mfma_f32_16x16x32_bf16).
//
// q.K^T: K rows are loaded straight into the A layout (lane l: row l%16,
// 8 elements per k-step), the group's queries are the B operand, and the C
// layout leaves head l%16's scores of rows 16*h + 4*(l/16) + j in lane l
// (h = 0, 1: the tile's two 16-row blocks).
//
// P.V: the weights stay where the softmax left them.  Lane l's eight
// weights (head l%16, rows 4*(l/16) + j and 16 + 4*(l/16) + j) are exactly
// its A operand once the 32 rows are taken in the order
// k = 8*q + e -> row 4*q + e (e < 4), 16 + 4*q + e - 4 (e >= 4).  V goes
// through a per-wave LDS tile and comes back with ds_read_b64_tr_b16 in
// that same row order as the B operand of each 16-column block; the output
// accumulates in the C layout (lane l: heads 4*(l/16) + r, column l%16 of
// the block).  Each weight is split into two bf16 terms (hi + lo, relative
// error about 2^-17) so the product keeps fp32-level accuracy.
template <class KV, int D, int G>
__device__ __forceinline__ void mf_compute(const DecodeArgs& a, int lane, int rs, int re,
                                           bool has_win, const MfRaw<KV, D>& raw,
                                           const bf16x8* qb, int w0, float sl,
                                           float sl2, float& m_c, float& l_c,
                                           f32x4 (&oacc)[D / 16], float* wls, uint16_t* vt) {
  constexpr int EPL = KV::kEpl;  // elements per 16-byte load
  constexpr int KPL = EPL / 8;    // MFMA k-steps per K load
  constexpr int LPR = D / EPL, RPI = 64 / LPR, T = kMfmaTile, UV = T / RPI, NK = D / 32;
  constexpr int NH = T / 16;  // 16-row MFMA blocks per tile
  constexpr int VROW = D + kVPad;
  static_assert(NH == 2, "the P.V row order assumes two 16-row blocks");
  const int lr = lane & 15, lq = lane >> 4, rg = lane / LPR, c = lane % LPR;
  const auto& kr = raw.k;
  const auto& vr = raw.v;
  f32x4 sc[NH];
#pragma unroll
  for (int h = 0; h < NH; ++h) {
    sc[h] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < NK; ++i)
      sc[h] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(KV::to_bf16(kr[h][i / KPL], i % KPL), qb[i],
                                                      sc[h], 0, 0, 0);
  }
  // Window logits go to LDS; the wave copies them out after its last tile
  // (a global store here would sit in the memory queue ahead of the waits
  // for this tile's and the next tile's data).
  if (has_win && lr < G) {
#pragma unroll
    for (int h = 0; h < NH; ++h)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = rs + 16 * h + 4 * lq + j;
        if (r < re) wls[lr * kMaxFusedSplitMfma + (r - a.Lp - w0)] = sc[h][j] * sl;
      }
  }
  // V rows of the tile into the wave's LDS tile, as bf16 (exact for fp8).
#pragma unroll
  for (int u = 0; u < UV; ++u)
#pragma unroll
    for (int hf = 0; hf < KPL; ++hf)
      *reinterpret_cast<bf16x8*>(vt + (u * RPI + rg) * VROW + c * EPL + 8 * hf) =
          KV::to_bf16(vr[u], hf);
  // Scores in log2 units, rounded once, so the largest one gets weight
  // exactly 1.
  float s2[NH][4];
  float mx = kNegBig;
#pragma unroll
  for (int h = 0; h < NH; ++h)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      s2[h][j] = rs + 16 * h + 4 * lq + j < re ? sc[h][j] * sl2 : kNegBig;
      mx = fmaxf(mx, s2[h][j]);
    }
  {
    float x1, x2;
    xor_pair<16>(mx, x1, x2);
    mx = fmaxf(x1, x2);
    xor_pair<32>(mx, x1, x2);
    mx = fmaxf(x1, x2);
  }
  const float mnew = fmaxf(m_c, mx);
  const float alpha = fast_exp2(m_c - mnew);
  m_c = mnew;
  l_c *= alpha;
  uint32_t ahi[4], alo[4];  // A operands: bf16 pairs of the weights (hi, lo)
#pragma unroll
  for (int h = 0; h < NH; ++h)
#pragma unroll
    for (int j = 0; j < 4; j += 2) {
      float p2[2];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        p2[t] = rs + 16 * h + 4 * lq + j + t < re ? fast_exp2(s2[h][j + t] - mnew) : 0.f;
        l_c += p2[t];
      }
      const uint32_t h0 = bf16_rne_bits(p2[0]), h1 = bf16_rne_bits(p2[1]);
      const uint32_t l0 = bf16_rne_bits(p2[0] - __uint_as_float(h0 << 16));
      const uint32_t l1 = bf16_rne_bits(p2[1] - __uint_as_float(h1 << 16));
      ahi[2 * h + j / 2] = h0 | (h1 << 16);
      alo[2 * h + j / 2] = l0 | (l1 << 16);
    }
  const bf16x8 a_hi = __builtin_bit_cast(bf16x8, make_uint4(ahi[0], ahi[1], ahi[2], ahi[3]));
  const bf16x8 a_lo = __builtin_bit_cast(bf16x8, make_uint4(alo[0], alo[1], alo[2], alo[3]));
  // The running output rows are heads 4*(l/16) + r; their rescale factors
  // live in lanes 4*(l/16) + r.
  float al[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) al[r] = __shfl(alpha, 4 * lq + r, 64);
#pragma unroll
  for (int cb = 0; cb < D / 16; ++cb)
#pragma unroll
    for (int r = 0; r < 4; ++r) oacc[cb][r] *= al[r];
  fence_wave();  // the V tile is written
  // Transposed reads: lane s of a 16-lane group points at row
  // 16*hh + 4*(l/16) + s/4, columns 16*cb + 4*(s%4) .. +3; lane n of the
  // group then holds rows 16*hh + 4*(l/16) + 0..3 of column 16*cb + n.
  const int s16 = lane & 15;
  const uint16_t* vsrc = vt + (4 * lq + (s16 >> 2)) * VROW + 4 * (s16 & 3);
#pragma unroll
  for (int cb = 0; cb < D / 16; ++cb) {
    const s16x4 b0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) s16x4*)(vsrc + 16 * cb));
    const s16x4 b1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) s16x4*)(vsrc + 16 * VROW + 16 * cb));
    const bf16x8 bv = __builtin_bit_cast(
        bf16x8, make_uint4(__builtin_bit_cast(uint32_t, __builtin_shufflevector(b0, b0, 0, 1)),
                           __builtin_bit_cast(uint32_t, __builtin_shufflevector(b0, b0, 2, 3)),
                           __builtin_bit_cast(uint32_t, __builtin_shufflevector(b1, b1, 0, 1)),
                           __builtin_bit_cast(uint32_t, __builtin_shufflevector(b1, b1, 2, 3))));
    oacc[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a_hi, bv, oacc[cb], 0, 0, 0);
    oacc[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a_lo, bv, oacc[cb], 0, 0, 0);
  }
  fence_wave();  // the next tile rewrites the V tile
}

// Dynamic LDS of the window logits of a sparse-mode split: G heads of at
// most max_fused_split rows (a multiple of 16 bytes).
__host__ __device__ constexpr uint32_t wl_lds_bytes(int G, bool mf) {
  return static_cast<uint32_t>(G) * max_fused_split(mf) * 4u;
}

// Dynamic LDS of an MFMA-tile workgroup of nw waves: the V tiles, then the
// per-wave partial results (their own space, so a wave writes its partials
// as soon as its last tile is done, without waiting for the others).  Each
// part is a multiple of 16 bytes.
template <int D>
__host__ __device__ constexpr uint32_t mf_vt_bytes(int nw) {
  return static_cast<uint32_t>(nw) * kMfmaTile * (D + kVPad) * 2;
}
template <int D, int G>
__host__ __device__ constexpr uint32_t mf_lds_bytes(int nw) {
  const uint32_t red = static_cast<uint32_t>(nw) * G * (D + 2) * 4;
  return mf_vt_bytes<D>(nw) + ((red + 15u) & ~15u);
}

template <class KV, int D, int G, int U, bool FUSED, bool KL, bool MF>
__device__ __forceinline__ void decode_body(const DecodeArgs& a) {
  constexpr int EPL = KV::kEpl;    // elements a lane loads per 16-byte access
  constexpr int LPR = D / EPL;     // lanes per row (V layout; K layout too without MF)
  constexpr int RPI = 64 / LPR;    // rows per load instruction
  constexpr int UU = MF ? U : unroll_for(G, D, KV::kBytes);  // loads in flight per operand
  constexpr int T = MF ? kMfmaTile : RPI * UU;      // rows per wave tile (<= 64)
  constexpr int NK = D / 32;       // MFMA k-steps per 16 rows (MF only)
  constexpr int KPL = EPL / 8;     // MFMA k-steps per K load (MF only)
  static_assert(T <= 64, "one kept position per lane");
  static_assert(!MF || G >= 2, "the MFMA tile serves grouped query heads");
  constexpr int KS = max_fused_split(MF);  // window rows of a sparse-mode split at most
  // The per-wave partial results (red): static LDS on the vector-ALU tile.
  // The MFMA tile keeps them in its dynamic LDS block (sized for the
  // launch's waves, mf_lds_bytes), after the per-wave V tiles.  The fused
  // step's skip bitmaps (one per wave) follow in dynamic LDS.
  constexpr int kRedBytes = MF ? 16 : kWaves * G * (D + 2) * 4;
  __shared__ __attribute__((aligned(16))) unsigned char smem[kRedBytes];
  extern __shared__ __attribute__((aligned(16))) unsigned char dyn_lds[];
  const int nw_launch = blockDim.x >> 6;
  const uint32_t mf_bytes = MF ? mf_lds_bytes<D, G>(nw_launch) : 0u;
  float (*red)[G][D + 2] =
      reinterpret_cast<float (*)[G][D + 2]>(MF ? dyn_lds + mf_vt_bytes<D>(nw_launch) : smem);
  __shared__ int kp_s[FUSED ? KS : 1];  // fused: kept positions of the split
  // MF: one V tile per wave (bf16, rows padded), read back transposed
  uint16_t* vt_w = reinterpret_cast<uint16_t*>(dyn_lds) + (threadIdx.x >> 6) * kMfmaTile * (D + kVPad);
  // Sparse mode: the split's window logits, head g at wl_s[g * KS + rank]
  // (dynamic LDS; none in dense mode).
  float* wl_s = reinterpret_cast<float*>(dyn_lds + mf_bytes);
  const uint32_t wl_bytes = a.mode != DSA_MODE_DENSE ? wl_lds_bytes(G, MF) : 0u;
  uint32_t* bm_all = reinterpret_cast<uint32_t*>(dyn_lds + mf_bytes + wl_bytes);

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int nwaves = blockDim.x >> 6;
  const int rg = lane / LPR;       // row group within the wave
  const int c = lane % LPR;        // EPL-element column chunk
  const int s = blockIdx.x % a.S;
  const int pair = blockIdx.x / a.S;
  const int kvh = pair % a.Hkv;
  const int b = pair / a.Hkv;

  // The workgroup's small per-(request, KV head) values do not depend on
  // one another, so they are loaded together, before anything uses them:
  // the decode position, the plan count or the stored skip count, the row
  // base and the fp8 scales.  An absent array is replaced by a readable
  // dummy address (the queries) and its value ignored, which keeps the
  // loads unconditional.  The stored skip offsets do not depend on the
  // decode position either: a wave that may own window rows loads them now
  // too, so the kept set is ready one memory latency sooner.
  // Queries first: their address depends on nothing loaded.
  uint4 qr[MF ? 1 : G][EPL / 8];
  if constexpr (!MF) {
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int hf = 0; hf < EPL / 8; ++hf)
        qr[g][hf] = *reinterpret_cast<const uint4*>(
            a.q + (static_cast<size_t>(b) * a.Hq + kvh * G + g) * D + (lane % LPR) * EPL + 8 * hf);
  }
  const int r0 = s * a.C;
  const int32_t* dummy32 = reinterpret_cast<const int32_t*>(a.q);
  const bool has_state = FUSED && a.state_cap > 0;
  const bool has_plan = !FUSED && a.mode != DSA_MODE_DENSE;
  const int t_raw = a.pos[b];
  const int cnt_raw = *(has_state ? a.st_count + pair : has_plan ? a.count + pair : dummy32);
  const int64_t rb_raw =
      *(a.row_base ? a.row_base + b : reinterpret_cast<const int64_t*>(a.q));
  // Scales exist only for fp8 caches (a bf16 call passes none).
  constexpr bool kScaled = KV::kBytes == 1;
  const float ks_raw = kScaled ? *(a.ks ? a.ks + pair : reinterpret_cast<const float*>(a.q)) : 1.f;
  const float vs_raw = kScaled ? *(a.vs ? a.vs + pair : reinterpret_cast<const float*>(a.q)) : 1.f;
  // Tiles of the split from its rows alone: the prompt tiles of an active
  // request (p0) and the most window tiles (wmax).  The wave-to-tile
  // mapping depends on these and not on the request's length, so the waves
  // that may rank window rows are known before the position arrives.  The
  // vector-ALU tile deals the tiles round robin; the MFMA tile gives each
  // wave a block of `per` consecutive tiles (prompt tiles first), so a wave
  // of prompt tiles issues its loads without waiting for a ranking.
  const int pe0 = min(r0 + a.C, a.Lp);
  const int p0 = pe0 > r0 ? (pe0 - r0 + T - 1) / T : 0;
  const int ws0 = max(r0, a.Lp);
  const int wmax = r0 + a.C > ws0 ? (r0 + a.C - ws0 + T - 1) / T : 0;
  const int per = MF ? (p0 + wmax + nwaves - 1) / nwaves : 0;
  // Fused step: the tags of the two kept lists (which numbers of skip
  // entries they belong to), and the lists themselves for the waves that
  // may own window rows.  Launches that keep no lists read a dummy address.
  const int2 tags_raw =
      FUSED && KL ? *reinterpret_cast<const int2*>(has_state
                                                 ? static_cast<const void*>(a.st_kc + 2 * pair)
                                                 : static_cast<const void*>(a.q))
            : make_int2(0, 0);
  PreRegs preld{};
  if constexpr (FUSED) {
    bool may_rank;
    if (per > 0) {
      const int jb0 = wave * per;
      may_rank = max(jb0, p0) < min(jb0 + per, p0 + wmax);
    } else {
      may_rank = p0 + ((wave - p0) % nwaves + nwaves) % nwaves < p0 + wmax;
    }
    load_pre<KL>(a, pair, lane, has_state && may_rank, preld);
  }
  // Settle the scalar values here, all at once: left alone, the compiler
  // sinks each load to its first use and waits for them one at a time.
  if constexpr (kScaled)
    asm volatile("" ::"s"(t_raw), "s"(cnt_raw), "s"(rb_raw), "s"(ks_raw), "s"(vs_raw));
  else
    asm volatile("" ::"s"(t_raw), "s"(cnt_raw), "s"(rb_raw));
  const RowRange rr = row_range_of<FUSED>(a, t_raw, cnt_raw);
  const int n = rr.n;
  if (s > 0 && r0 >= n) return;
  const int r1 = min(n, r0 + a.C);
  const int nsplit = (n + a.C - 1) / a.C;
  const bool dense = a.mode == DSA_MODE_DENSE;
  const int w0 = max(r0, a.Lp) - a.Lp;  // first window rank of the split

  // Byte offset of this lane's first element (strides arrive in bytes).
  constexpr int E = KV::kBytes;
  const int64_t base = (a.row_base ? rb_raw * E : static_cast<int64_t>(b) * a.sb) +
                       static_cast<int64_t>(kvh) * a.sh + c * EPL * E;
  const uint8_t* kb = a.k + base;
  const uint8_t* vb = a.v + base;
  // fp8 caches: the K scale folds into the logit scale, the V scale into
  // the final normalisation (both 1 for bf16).
  const float sl = kScaled && a.ks ? a.scale * ks_raw : a.scale;
  const float sl2 = kScaled && a.ks ? a.scale_log2 * ks_raw : a.scale_log2;
  const int32_t* widx = FUSED ? nullptr : a.idx + static_cast<size_t>(pair) * a.plan_cap - a.Lp;

  // MFMA operands: K in the A layout (lane l: row l%16; k-step i takes the
  // 8 elements 32*KPL*(i/KPL) + EPL*(l/16) + 8*(i%KPL) .. +7, so one 16-byte
  // load serves KPL k-steps), q^T in the B layout (lane l: query head l%16
  // of the group, the same elements; zero for l%16 >= G).
  const int lr = lane & 15, lq = lane >> 4;
  const uint8_t* kmf = a.k + (base - c * EPL * E) + EPL * E * lq;
  bf16x8 qb[MF ? NK : 1];
  if constexpr (MF) {
#pragma unroll
    for (int i = 0; i < NK; ++i) {
      uint4 x = make_uint4(0, 0, 0, 0);
      if (lr < G)
        x = *reinterpret_cast<const uint4*>(
            a.q + (static_cast<size_t>(b) * a.Hq + kvh * G + lr) * D +
            32 * KPL * (i / KPL) + EPL * lq + 8 * (i % KPL));
      qb[i] = __builtin_bit_cast(bf16x8, x);
    }
  }

  // Ring layouts: the start of the lap that holds position t (in positions
  // after the sinks), for the slot arithmetic of the window tiles.
  const int ring_lap = (a.ring && rr.t >= a.Ns) ? (rr.t - a.Ns) / a.ring * a.ring : 0;

  // Tiles never straddle the prompt/decode boundary: the split's prompt rows
  // [r0, pe) and decode rows [wst, r1) are each cut into tiles of T rows,
  // tile j going to wave j % nwaves.  Prompt tiles and dense-mode decode
  // tiles load at once; diagonal-mode decode tiles wait for their kept
  // positions.  (Both modes cut the same way, so with nothing skipped they
  // add the same numbers in the same order.)
  const int pe = min(r1, a.Lp);
  const int wst = max(r0, a.Lp);
  const int P = pe > r0 ? (pe - r0 + T - 1) / T : 0;
  const int Wn = r1 > wst ? (r1 - wst + T - 1) / T : 0;

  SkipSet ss{};
  // The wave holding window rank 0 (the first decode tile of the pair)
  // reports the plan's count and flags, as dsa_plan would.
  bool reporter = false;
  int rep_flags = 0;
  // The wave's tiles: j = jb, jb + js, ... below je (see p0 and per; an
  // active request has P == p0 and at most wmax window tiles).
  const int ntile = P + Wn;
  int jb = wave, je = ntile, js = nwaves;
  if (per > 0) {
    jb = min(wave * per, ntile);
    je = min(jb + per, ntile);
    js = 1;
  }
  // First window tile of the wave (it has one if jw0 < je).
  const int jw0 = js == 1 ? max(jb, P) : P + ((wave - P) % nwaves + nwaves) % nwaves;
  if constexpr (FUSED)
    reporter = rr.t < 0 ? (s == 0 && wave == 0) : (w0 == 0 && Wn > 0 && jw0 == P && jw0 < je);

  // Rows [rs, re) of tile j of the split and, for a window tile, the kept
  // position of row rs + i in lane i (after the ranking, for the fused step).
  struct TileRows {
    int rs, re;
    bool has_win;
    int pos_l;
  };
  auto rows_of = [&](int j) {
    TileRows tr;
    const bool dec = j >= P;
    tr.has_win = dec && !dense;
    tr.rs = dec ? wst + (j - P) * T : r0 + j * T;
    tr.re = min(tr.rs + T, dec ? r1 : pe);
    tr.pos_l = 0;
    if (tr.has_win) {
      if constexpr (FUSED) {
        if (lane < tr.re - tr.rs) tr.pos_l = kp_s[tr.rs + lane - a.Lp - w0];
      } else {
        if (lane < tr.re - tr.rs) tr.pos_l = min(max(widx[tr.rs + lane], 0), rr.t);
      }
      if (a.ring && tr.pos_l >= a.Ns) {  // ring slot: (pos - S) mod ring, after the S sinks
        // kept positions lie in (t - ring, t], so one conditional add
        // reduces them from the lap of t (a position outside that range
        // only comes from a corrupt plan: it reads slot 0)
        int sl = tr.pos_l - a.Ns - ring_lap;
        if (sl < 0) sl += a.ring;
        tr.pos_l = a.Ns + max(sl, 0);
      }
    }
    return tr;
  };

  // Fused step, vector-ALU tile: a wave whose first tile holds prompt rows
  // issues that tile's K loads before the ranking below, so they are in
  // flight while the window rows are ranked (V too would not fit in 128
  // registers).  The MFMA tile ranks first: its waves of prompt tiles have
  // nothing to rank, and a wave that issued a tile's loads ahead of its
  // ranking would stall at issue behind the CU's full memory queue and rank
  // late.
  constexpr bool kHoist = FUSED && !MF;
  typename KV::Raw kr[UU], vr[UU];  // the vector-ALU tile's K/V
  const bool pre = kHoist && wave < P;
  MfRaw<KV, D> ra, rb;  // the MFMA tile's K/V: two tiles in flight
  if constexpr (kHoist) {
    if (pre) {
      const int rs = r0 + wave * T;
      const int re = min(rs + T, pe);
#pragma unroll
      for (int u = 0; u < UU; ++u) {
        const int r = rs + u * RPI + rg;
        const int cr = r < re ? r : 0;  // rows past the tile end read row 0, weight 0
        kr[u] = KV::load(kb + cr * a.sr);
      }
    }
  }
  bool from_list = false;
  if constexpr (FUSED) {
    // Each wave finds the kept window rows of its own tiles (its own slice
    // of kp_s).  From the stored kept list when it matches this step: the
    // list for k skip entries sits in slot k % 2 tagged k + 1 (phase 2 and
    // 3, k >= 1).  Otherwise (phase 1, the first selection step, or a state
    // whose list is missing) from a skip bitmap of the stored offsets in
    // the wave's own LDS slice.
    const int kneed = min(rr.t - (a.Natt - 1), a.state_cap);
    from_list = KL && has_state && kneed >= 1 &&
                ((kneed & 1) ? tags_raw.y : tags_raw.x) == kneed + 1 && cnt_raw >= kneed;
    if (from_list) {
      const int sl = kneed & 1;
      const uint16_t* list =
          a.st_kept + (static_cast<size_t>(pair) * 2 + sl) * ((a.kept_cap + 1) & ~1);
      for (int j = jw0; j < je; j += js) {
        const int lo = wst + (j - P) * T - a.Lp;
        const int hi = min(lo + a.Lp + T, r1) - a.Lp;
        for (int r = lo + lane; r < min(hi, a.Ns); r += 64) kp_s[r - w0] = r;  // sinks
#pragma unroll
        for (int i = 0; i < kPre / 2; ++i) {
          const uint32_t w0v = preld.w[i], w1v = preld.w[kPre / 2 + i];
          const int d = static_cast<int>(sl ? w1v : w0v);
          const int e = lane + 64 * i;
          const int r = a.Ns + e;
          if (e < a.kept_cap && r >= lo && r < hi) kp_s[r - w0] = rr.t - d;
        }
        // entries past the ones loaded ahead (lists longer than 32 * kPre)
        const int e_hi = min(a.kept_cap, hi - a.Ns);
        for (int e = max(32 * kPre, lo - a.Ns) + lane; e < e_hi; e += 64)
          kp_s[a.Ns + e - w0] = rr.t - static_cast<int>(list[e]);
      }
      fence_wave();
    } else {
      if (jw0 < je) {
        build_skip_set<KL>(a, pair, lane, rr.t, has_state ? cnt_raw : 0, bm_all + wave * a.words,
                       preld, ss);
      }
      for (int j = jw0; j < je; j += js) {
        const int rs = wst + (j - P) * T;
        const int re = min(rs + T, r1);
        rank_window(lane, ss, rs - a.Lp, re - a.Lp, kp_s, w0);
      }
    }
    // The reporting wave settles the plan flags now, so the skip set is not
    // live through the K/V loop (a kept list has the right count by
    // construction).
    if (reporter) {
      rep_flags = rr.flags;
      if (rr.t >= 0 && !from_list) {
        rep_flags |= ss.flags;
        const int kept = count_kept(ss, lane);
        if (!(ss.flags & (DSA_FLAG_STATE_BEHIND | DSA_FLAG_BAD_OFFSET)) &&
            kept != min(rr.t + 1, a.Natt))
          rep_flags |= DSA_FLAG_COUNT;
      }
    }
    // Vector-ALU tile: the prompt waves' V loads (and later tiles) wait until
    // the window rows are ranked, so the window rows' loads enter each CU's
    // memory queue ahead of the prompt V traffic instead of behind all of
    // it; the hoisted prompt K loads keep the memory busy meanwhile.  (As
    // compiled, a prompt wave also waits for its hoisted K rows before this
    // barrier: the loop preheader of the ranking waits for the stored
    // offsets with a vmcnt that, after the conditional hoisted loads, must
    // count all of them.  Issuing its V loads earlier measured slower.)
    if constexpr (!MF) {
      if (Wn > 0 && P > 0) __syncthreads();
    }
  }

  float qf[MF ? 1 : G][EPL];
  float m[G], l[G], acc[G][EPL];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    if constexpr (!MF) {
#pragma unroll
      for (int hf = 0; hf < EPL / 8; ++hf) {
        float f8[8];
        unpack8(qr[g][hf], f8);
#pragma unroll
        for (int e = 0; e < 8; ++e) qf[g][8 * hf + e] = f8[e];
      }
    }
    m[g] = kNegBig;
    l[g] = 0.f;
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[g][e] = 0.f;
  }
  float m_c = kNegBig, l_c = 0.f;  // MF: running max / partial sum of head lr
  f32x4 oacc[MF ? D / 16 : 1];     // MF: output, C layout (heads x 16 columns per block)
#pragma unroll
  for (int cb = 0; cb < (MF ? D / 16 : 1); ++cb) oacc[cb] = f32x4{0.f, 0.f, 0.f, 0.f};

  // One vector-ALU tile of the wave (tile j of the split).  hoisted: its K
  // rows were loaded before the ranking.
  auto tile = [&](int j, bool hoisted) {
    const TileRows tr = rows_of(j);
    const int rs = tr.rs, re = tr.re, pos_l = tr.pos_l;
    const bool has_win = tr.has_win;
#pragma unroll
    for (int u = 0; u < UU; ++u) {
      const int r = rs + u * RPI + rg;
      const int wpos = has_win ? __shfl(pos_l, u * RPI + rg, 64) : 0;
      int cr = 0;  // rows past the tile end read row 0 and get weight 0
      if (r < re) cr = has_win ? a.Lp + wpos : r;
      if (!hoisted) kr[u] = KV::load(kb + cr * a.sr);
      vr[u] = KV::load(vb + cr * a.sr);
    }
    // Every load of the tile is issued before any arithmetic on it.
    __builtin_amdgcn_sched_barrier(0);

    float sc[UU][G];
#pragma unroll
    for (int u = 0; u < UU; ++u) {
      float kf[EPL];
      KV::widen(kr[u], kf);
#pragma unroll
      for (int g = 0; g < G; ++g) {
        float x = 0.f;
#pragma unroll
        for (int e = 0; e < EPL; ++e) x = fmaf(qf[g][e], kf[e], x);
        sc[u][g] = group_sum<LPR>(x);
      }
    }
    // Window logits go to LDS (copied out after the wave's last tile, so
    // no global store waits ahead of this tile's V data).
    if (has_win && c == 0) {
#pragma unroll
      for (int u = 0; u < UU; ++u) {
        const int r = rs + u * RPI + rg;
        if (r < re) {
#pragma unroll
          for (int g = 0; g < G; ++g) wl_s[g * KS + (r - a.Lp - w0)] = sc[u][g] * sl;
        }
      }
    }
#pragma unroll
    for (int g = 0; g < G; ++g) {
      // Scores in log2 units, rounded once, so the largest one gets weight
      // exactly 1.
      float mx = kNegBig;
#pragma unroll
      for (int u = 0; u < UU; ++u) {
        sc[u][g] = rs + u * RPI + rg < re ? sc[u][g] * sl2 : kNegBig;
        mx = fmaxf(mx, sc[u][g]);
      }
      const float mnew = fmaxf(m[g], mx);
      const float alpha = fast_exp2(m[g] - mnew);
      m[g] = mnew;
      l[g] *= alpha;
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[g][e] *= alpha;
    }
#pragma unroll
    for (int u = 0; u < UU; ++u) {
      float vf[EPL];
      KV::widen(vr[u], vf);
      const bool ok = rs + u * RPI + rg < re;
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float p = ok ? fast_exp2(sc[u][g] - m[g]) : 0.f;
        l[g] += p;
#pragma unroll
        for (int e = 0; e < EPL; ++e) acc[g][e] = fmaf(p, vf[e], acc[g][e]);
      }
    }
  };
  if constexpr (MF) {
    // The wave's block of tiles two at a time: tiles j and j + 1 are both
    // in flight before either is computed (each branch is straight-line
    // code, so the wait for the first tile does not also wait for the
    // second).
    auto compute = [&](const TileRows& tr, const MfRaw<KV, D>& raw) {
      mf_compute<KV, D, G>(a, lane, tr.rs, tr.re, tr.has_win, raw, qb, w0, sl, sl2, m_c, l_c,
                           oacc, wl_s, vt_w);
    };
    for (int j = jb; j < je; j += 2 * js) {
      const TileRows ta = rows_of(j);
      mf_load<KV, D>(a, lane, ta.rs, ta.re, ta.has_win, ta.pos_l, kmf, vb, ra);
      const int j2 = j + js;
      if (j2 < je) {
        const TileRows tb = rows_of(j2);
        mf_load<KV, D>(a, lane, tb.rs, tb.re, tb.has_win, tb.pos_l, kmf, vb, rb);
        compute(ta, ra);
        compute(tb, rb);
      } else {
        compute(ta, ra);
      }
    }
  } else {
    // A wave with hoisted K loads runs its first tile outside the loop, so
    // the loop's registers never overlap loads still in flight.
    int j = wave;
    if (kHoist && pre) {
      tile(j, true);
      j += nwaves;
    }
    for (; j < P + Wn; j += nwaves) tile(j, false);
  }

  if constexpr (FUSED) {
    if (reporter && lane == 0) {
      a.plan_count[pair] = rr.t < 0 ? 0 : n - a.Lp;
      a.plan_flags[pair] = rep_flags;
    }
  }

  if constexpr (MF) {
    // Head g's running max sits in the lanes with lr == g; its sum is split
    // over the four lanes lr + 16*q.  The output is already the wave's full
    // sum in the C layout: lane l holds heads 4*(l/16) + r, column l%16 of
    // each 16-column block.
    float x1, x2;
    xor_pair<16>(l_c, x1, x2);
    float lt = x1 + x2;
    xor_pair<32>(lt, x1, x2);
    lt = x1 + x2;
#pragma unroll
    for (int cb = 0; cb < D / 16; ++cb)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        if (4 * lq + r < G) red[wave][4 * lq + r][16 * cb + lr] = oacc[cb][r];
    if (lane < G) {
      red[wave][lane][D] = m_c;
      red[wave][lane][D + 1] = lt;
    }
  }
  // Merge the row groups of the wave (lanes c, c + LPR, c + 2*LPR, ...).
  if constexpr (!MF) {
    if constexpr (LPR <= 4) merge_groups<4, G, EPL>(m, l, acc);
    if constexpr (LPR <= 8) merge_groups<8, G, EPL>(m, l, acc);
    merge_groups<16, G, EPL>(m, l, acc);
    merge_groups<32, G, EPL>(m, l, acc);
  }
  if (!MF && rg == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
#pragma unroll
      for (int e = 0; e < EPL; ++e) red[wave][g][c * EPL + e] = acc[g][e];
      if (c == 0) {
        red[wave][g][D] = m[g];
        red[wave][g][D + 1] = l[g];
      }
    }
  }
  __syncthreads();

  // Phase-2 selection, when this workgroup saw every kept window key (the
  // same for every wave of the workgroup).  The sinks (the first Ns kept
  // ranks) are never candidates.  The stored count is the one loaded at the
  // start (only this workgroup writes it), so the selection waits for no
  // memory.
  bool sel = false;
  const int ksel = rr.t - (a.Natt - 1);
  const int nwin = n - a.Lp - a.Ns;
  float* const wl_win = wl_s + a.Ns;  // head g's window logits at wl_win[g * KS + j]
  if constexpr (FUSED) {
    sel = nsplit == 1 && rr.t >= a.Natt - 1 && rr.t <= a.Nr + a.Ns - 2 && ksel < a.state_cap;
    if (sel && cnt_raw < ksel) {
      if (wave == nwaves - 1 && lane == 0) a.st_flags[pair] |= DSA_FLAG_STATE_BEHIND;
      sel = false;
    }
  }
  // Stores of window logits and plan rows wait until every wave has left
  // its tile loop, so none sits in the memory queue ahead of a wait for K/V
  // data.  Head g's window logits (split ranks w0 ..) are copied out by wave
  // nwaves - 1 - g (and so on round the waves), which then, for grouped
  // heads, turns them into the head's window softmax for the selection,
  // while the first waves merge the outputs below.  The last wave copies
  // the plan rows.
  const int nws = r1 > wst ? r1 - wst : 0;  // window rows of the split
  for (int g = nwaves - 1 - wave; g < G; g += nwaves) {
    if (a.wlog && !dense) {
      float* dst = a.wlog + (static_cast<size_t>(b) * a.Hq + kvh * G + g) * a.plan_cap + w0;
      for (int i = lane; i < nws; i += 64) dst[i] = wl_s[g * KS + i];
    }
    if constexpr (FUSED && G > 1) {
      if (sel) head_terms(lane, nwin, wl_win + g * KS);
    }
  }
  if constexpr (FUSED) {
    if (wave == nwaves - 1) {
      int32_t* plan = a.plan_idx + static_cast<size_t>(pair) * a.plan_cap + w0;
      for (int i = lane; i < nws; i += 64) plan[i] = kp_s[i];
    }
  }
  // Merge the waves: wave w takes query heads w, w + nwaves, ... of the
  // group, and lane j columns j and j + 64.  Every LDS read of a head is
  // issued before the first is used, with no branches: slots past the
  // workgroup's waves read its last wave again (the maximum does not
  // change) and add nothing (the waves are added in order).
  constexpr int NWM = MF ? kWavesMfma : kWaves;  // waves of a workgroup at most
  for (int g = wave; g < G; g += nwaves) {
    float mw[NWM], lw[NWM], a0[NWM], a1[NWM];
#pragma unroll
    for (int w = 0; w < NWM; ++w) {
      const int wr = min(w, nwaves - 1);
      mw[w] = red[wr][g][D];
      lw[w] = red[wr][g][D + 1];
      a0[w] = red[wr][g][lane];
      a1[w] = D == 128 ? red[wr][g][(lane + 64) % D] : 0.f;
    }
    float M = kNegBig;
#pragma unroll
    for (int w = 0; w < NWM; ++w) M = fmaxf(M, mw[w]);
    float L = 0.f, A0 = 0.f, A1 = 0.f;
#pragma unroll
    for (int w = 0; w < NWM; ++w) {
      const bool ok = w < nwaves;
      const float sw = fast_exp2(mw[w] - M);
      L = ok ? fmaf(lw[w], sw, L) : L;
      A0 = ok ? fmaf(a0[w], sw, A0) : A0;
      if constexpr (D == 128) A1 = ok ? fmaf(a1[w], sw, A1) : A1;
    }
    const int h = kvh * G + g;
    if (nsplit <= 1) {
      float inv = L > 0.f ? 1.f / L : 0.f;
      if (kScaled && a.vs) inv *= vs_raw;
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

  if constexpr (FUSED) {
    if constexpr (G > 1) {
      if (sel) __syncthreads();  // every head's terms are in LDS
    }
    if (sel && wave == nwaves - 1) {
      int jbest;
      if constexpr (G > 1)
        jbest = terms_argmin<G>(lane, nwin, [&](int g, int j) { return wl_win[g * KS + j]; });
      else
        jbest = window_argmin<1>(lane, nwin, [&](int, int j) { return wl_win[j]; });
      if (jbest < 0 || jbest >= nwin) jbest = 0;  // only for NaN logits
      if (lane == 0) {
        const int d = min(max(rr.t - kp_s[a.Ns + jbest], 0), a.Nr - 2);
        a.st_off[static_cast<size_t>(pair) * a.state_cap + ksel] = static_cast<uint16_t>(d);
        a.st_count[pair] = ksel + 1;
      }
      // The kept list of the next step, into the other slot.
      if (KL && nwin == a.kept_cap) {
        const int sl = (ksel + 1) & 1;
        write_kept_list(lane, nwin, jbest, rr.t, a.Natt - a.Ns + ksel,
                        [&](int r) { return kp_s[a.Ns + r]; },
                        a.st_kept + (static_cast<size_t>(pair) * 2 + sl) * ((a.kept_cap + 1) & ~1),
                        a.st_kc + 2 * pair + sl, ksel + 1);
      }
    }
  }
}

// One query head per KV head: four waves per SIMD stay resident (at most
// 128 registers), so a small sparse layer runs as a single round of
// workgroups.  (Larger groups keep their accumulators in registers instead.)
template <class KV, int D, int G, int U, bool FUSED, bool KL>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(G == 1 ? 4 : 1, 8)))
void decode_kernel(DecodeArgs a) {
  decode_body<KV, D, G, U, FUSED, KL, false>(a);
}

// The grouped-head (MFMA) tile holds K and V of two 32-row tiles and the
// output blocks in registers (up to 256 of them: two waves per SIMD).
template <class KV, int D, int G, bool FUSED, bool KL>
__global__ __launch_bounds__(64 * kWavesMfma) __attribute__((amdgpu_waves_per_eu(2, 8)))
void decode_mfma_kernel(DecodeArgs a) {
  decode_body<KV, D, G, 2, FUSED, KL, true>(a);
}

// out = sum_s e^{m_s - M} acc_s / sum_s e^{m_s - M} l_s over the splits of
// (request b, query head g of KV head kvh), in base-2 exponents (the partial
// maxima are kept in log2 units).  Called by one wave.
template <int D>
__device__ __forceinline__ void combine_one(const DecodeArgs& a, int lane, int b, int kvh, int g,
                                            int G, int nsplit) {
  const int pair = b * a.Hkv + kvh;
  const float* pp = a.part + (static_cast<size_t>(pair) * a.S * G + g) * (D + 2);
  const size_t sstride = static_cast<size_t>(G) * (D + 2);
  // Maxima and sums: one split per lane.
  float M = kNegBig;
  for (int s = lane; s < nsplit; s += 64) M = fmaxf(M, pp[s * sstride + D]);
  M = wave_max(M);
  float L = 0.f;
  for (int s = lane; s < nsplit; s += 64)
    L = fmaf(pp[s * sstride + D + 1], fast_exp2(pp[s * sstride + D] - M), L);
  L = wave_sum(L);
  // Weighted rows: lanes over columns, eight splits' loads in flight.
  float A0 = 0.f, A1 = 0.f;
  for (int s0 = 0; s0 < nsplit; s0 += 64) {
    const int sl = s0 + lane;
    const float w = sl < nsplit ? fast_exp2(pp[sl * sstride + D] - M) : 0.f;
    const int n = min(64, nsplit - s0);
    for (int j0 = 0; j0 < n; j0 += 8) {
      float x0[8], x1[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int sj = s0 + min(j0 + j, n - 1);
        x0[j] = pp[sj * sstride + lane];
        if constexpr (D == 128) x1[j] = pp[sj * sstride + lane + 64];
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float sw = j0 + j < n ? __shfl(w, j0 + j, 64) : 0.f;
        A0 = fmaf(x0[j], sw, A0);
        if constexpr (D == 128) A1 = fmaf(x1[j], sw, A1);
      }
    }
  }
  float inv = L > 0.f ? 1.f / L : 0.f;
  if (a.vs) inv *= a.vs[pair];
  float* o = a.out + (static_cast<size_t>(b) * a.Hq + kvh * G + g) * D;
  o[lane] = A0 * inv;
  if constexpr (D == 128) o[lane + 64] = A1 * inv;
}

// One wave per (request, query head).
template <int D>
__global__ __launch_bounds__(kBlock) void combine_kernel(DecodeArgs a, int G) {
  const int lane = threadIdx.x & 63;
  const int bh = blockIdx.x * kWaves + (threadIdx.x >> 6);
  if (bh >= a.B * a.Hq) return;
  const int b = bh / a.Hq;
  const int h = bh % a.Hq;
  const RowRange rr = row_range<false>(a, b, b * a.Hkv + h / G);
  const int nsplit = (rr.n + a.C - 1) / a.C;
  if (nsplit <= 1) return;
  combine_one<D>(a, lane, b, h / G, h % G, G, nsplit);
}

// Fused step, several splits: one workgroup per (request, KV head).  Its
// first min(G, 4) waves merge the splits of the group's query heads while
// one more wave runs the phase-2 selection on the window logits and the plan
// the split workgroups wrote (the selection does not depend on the merged
// outputs, so the two run side by side).
constexpr int kCombineWaves = kWaves;

template <int D, int G>
__global__ __launch_bounds__(kBlock + 64) void combine_select_kernel(DecodeArgs a) {
  constexpr int CW = G < kCombineWaves ? G : kCombineWaves;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int pair = blockIdx.x;
  const int b = pair / a.Hkv;
  const int kvh = pair % a.Hkv;
  const RowRange rr = row_range<true>(a, b, pair);
  const int nsplit = (rr.n + a.C - 1) / a.C;
  if (nsplit <= 1) return;
  if (wave < CW) {
    for (int g = wave; g < G; g += CW) combine_one<D>(a, lane, b, kvh, g, G, nsplit);
    return;
  }
  const int t = rr.t;
  if (t < a.Natt - 1 || t > a.Nr + a.Ns - 2) return;
  const int k = t - (a.Natt - 1);
  if (k >= a.state_cap) return;
  const int cnt = a.st_count[pair];
  if (cnt < k) {
    if (lane == 0) a.st_flags[pair] |= DSA_FLAG_STATE_BEHIND;
    return;
  }
  const int nwin = rr.n - a.Lp - a.Ns;  // window keys after the sinks
  const float* wl = a.wlog + (static_cast<size_t>(b) * a.Hq + kvh * G) * a.plan_cap + a.Ns;
  const int plan_cap = a.plan_cap;
  int jbest = window_argmin<G>(lane, nwin, [&](int g, int j) { return wl[g * plan_cap + j]; });
  if (jbest < 0 || jbest >= nwin) jbest = 0;  // only for NaN logits
  const int32_t* kept_pos = a.plan_idx + static_cast<size_t>(pair) * a.plan_cap + a.Ns;
  if (lane == 0) {
    const int d = min(max(t - kept_pos[jbest], 0), a.Nr - 2);
    a.st_off[static_cast<size_t>(pair) * a.state_cap + k] = static_cast<uint16_t>(d);
    a.st_count[pair] = k + 1;
  }
  if (a.kept_read && nwin == a.kept_cap) {
    const int sl = (k + 1) & 1;
    write_kept_list(lane, nwin, jbest, t, a.Natt - a.Ns + k, [&](int r) { return kept_pos[r]; },
                    a.st_kept + (static_cast<size_t>(pair) * 2 + sl) * ((a.kept_cap + 1) & ~1),
                    a.st_kc + 2 * pair + sl, k + 1);
  }
}

template <class KV, int D, int G, int U, bool FUSED, bool KL, bool MF>
void launch_split(const Derived& d, const DecodeArgs& a, hipStream_t st, hipEvent_t t0,
                  hipEvent_t t1) {
  const int grid = d.B * d.Hkv * d.S;
  const int nw = KV::kBytes == 1 ? d.NW_fp8 : d.NW;
  const int block = 64 * nw;
  const uint32_t lds = (MF ? mf_lds_bytes<D, G>(nw) : 0u) +
                       (a.mode != DSA_MODE_DENSE ? wl_lds_bytes(G, MF) : 0u) +
                       (FUSED ? static_cast<uint32_t>(sizeof(uint32_t) * nw * a.words) : 0u);
  if constexpr (MF) {
    if (t0 || t1)
      hipExtLaunchKernelGGL(decode_mfma_kernel<KV, D, G, FUSED, KL>, dim3(grid), dim3(block), lds,
                            st, t0, t1, 0, a);
    else
      decode_mfma_kernel<KV, D, G, FUSED, KL><<<grid, block, lds, st>>>(a);
  } else {
    if (t0 || t1)
      hipExtLaunchKernelGGL(decode_kernel<KV, D, G, U, FUSED, KL>, dim3(grid), dim3(block), lds,
                            st, t0, t1, 0, a);
    else
      decode_kernel<KV, D, G, U, FUSED, KL><<<grid, block, lds, st>>>(a);
  }
}

template <class KV, int D, int G, bool FUSED, bool KL>
hipError_t launch_dg(const Derived& d, const DecodeArgs& a, hipStream_t st, hipEvent_t t0,
                     hipEvent_t t1) {
  // With several splits the stop event goes to the combine, so a timed call
  // covers every kernel it launches.
  const bool split = d.S > 1;
  if constexpr (uses_mfma_tile(G))
    launch_split<KV, D, G, 2, FUSED, KL, true>(d, a, st, t0, split ? nullptr : t1);
  else
    launch_split<KV, D, G, unroll_of(G), FUSED, KL, false>(d, a, st, t0, split ? nullptr : t1);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !split) return e;
  if (FUSED) {
    constexpr int cw = G < kCombineWaves ? G : kCombineWaves;
    if (t1)
      hipExtLaunchKernelGGL(combine_select_kernel<D, G>, dim3(d.B * d.Hkv), dim3(64 * (cw + 1)), 0,
                            st, nullptr, t1, 0, a);
    else
      combine_select_kernel<D, G><<<d.B * d.Hkv, 64 * (cw + 1), 0, st>>>(a);
  } else {
    const int cgrid = (d.B * d.Hq + kWaves - 1) / kWaves;
    if (t1)
      hipExtLaunchKernelGGL(combine_kernel<D>, dim3(cgrid), dim3(kBlock), 0, st, nullptr, t1, 0, a,
                            G);
    else
      combine_kernel<D><<<cgrid, kBlock, 0, st>>>(a, G);
  }
  return hipGetLastError();
}

template <class KV, int D, bool FUSED, bool KL>
hipError_t launch_d(const Derived& d, const DecodeArgs& a, hipStream_t st, hipEvent_t t0,
                    hipEvent_t t1) {
  switch (d.G) {
    case 1: return launch_dg<KV, D, 1, FUSED, KL>(d, a, st, t0, t1);
    case 2: return launch_dg<KV, D, 2, FUSED, KL>(d, a, st, t0, t1);
    case 4: return launch_dg<KV, D, 4, FUSED, KL>(d, a, st, t0, t1);
    default: return launch_dg<KV, D, 8, FUSED, KL>(d, a, st, t0, t1);
  }
}

// Every kernel of one K/V element type: the decode kernel (plain or fused
// step) for the call's head_dim, then the combine when a request is split.
template <class KV>
hipError_t launch_kv(const Derived& d, const DecodeArgs& a, hipStream_t st, hipEvent_t t0,
                     hipEvent_t t1, bool fused) {
  // The fused step has two builds: with the kept lists of the selection
  // state (launch rule kept_read) and without, so launches that keep no
  // lists carry none of their code.
  if (fused && a.kept_read)
    return d.D == 64 ? launch_d<KV, 64, true, true>(d, a, st, t0, t1)
                     : launch_d<KV, 128, true, true>(d, a, st, t0, t1);
  if (fused)
    return d.D == 64 ? launch_d<KV, 64, true, false>(d, a, st, t0, t1)
                     : launch_d<KV, 128, true, false>(d, a, st, t0, t1);
  return d.D == 64 ? launch_d<KV, 64, false, false>(d, a, st, t0, t1)
                   : launch_d<KV, 128, false, false>(d, a, st, t0, t1);
}

}  // namespace
}  // namespace dsa

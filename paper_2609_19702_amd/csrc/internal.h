// Internal declarations shared by the library's translation units: the
// derived launch configuration, the kernel argument blocks and the launchers.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "dsa.h"

namespace dsa {

// Everything a call needs, derived once from (params, shape) on the host.
struct Derived {
  int B, Hq, Hkv, G, D;
  int Lp, Ldec, Natt, mode;
  int Ns;         // sink positions kept ahead of the window (0 in dense mode)
  int Nr;         // window W after the sinks: N_r (diagonal), N_att - S (window mode)
  int plan_cap;   // kept decode rows per (request, KV head): min(N_att, L_dec), 0 when dense
  int state_cap;  // skip entries per (request, KV head): W - (N_att - S) in diagonal mode, else 0
  int words;      // 32-bit words of a skip bitmap over W offsets (0 without a state)
  dsa_plan_layout plan;
  dsa_state_layout state;
  int rows_max;   // prompt rows + the most decode rows one request can attend
  int U;          // loads in flight per wave per operand (unroll_of(G))
  int C;          // rows per split workgroup
  int S;          // splits per (request, KV head), upper bound
  int NW;         // waves per decode workgroup (1..kWaves), bf16 caches
  int NW_fp8;     // the same for fp8 caches (tiles of twice the rows)
  bool MF;        // grouped query heads on the MFMA tile (uses_mfma_tile(G))
  int kept_read;  // 1: selections store kept lists and the fused step reads its kept rows from them
  size_t ws_bytes;
};

dsa_status derive(const dsa_params* p, const dsa_shape* s, Derived* d);

// Launch-shape choices, measured on MI355X and fixed at build time: a call's
// launch configuration and workspace size depend only on its parameters and
// shape.  A tuning build may override any of them with -D.
#ifndef DSA_TUNE_SPLIT_KB
#define DSA_TUNE_SPLIT_KB 192  // K+V bytes per split workgroup, sparse modes, vector-ALU tile
#endif
#ifndef DSA_TUNE_SPLIT_KB_MFMA
#define DSA_TUNE_SPLIT_KB_MFMA 256  // the same for the grouped-head MFMA tile
#endif
#ifndef DSA_TUNE_SPLIT_KB_DENSE_64
#define DSA_TUNE_SPLIT_KB_DENSE_64 24  // dense mode, d = 64, one query head per KV head
#endif
#ifndef DSA_TUNE_SPLIT_KB_DENSE_128
#define DSA_TUNE_SPLIT_KB_DENSE_128 96  // dense mode, d = 128, one query head per KV head
#endif
#ifndef DSA_TUNE_SPLIT_KB_DENSE_MFMA
#define DSA_TUNE_SPLIT_KB_DENSE_MFMA 128  // dense mode, grouped query heads
#endif
#ifndef DSA_TUNE_MIN_WGS
#define DSA_TUNE_MIN_WGS 512  // split further while a launch has fewer workgroups (dense mode)
#endif
#ifndef DSA_TUNE_MIN_WGS_SPARSE
#define DSA_TUNE_MIN_WGS_SPARSE 256  // the same in the sparse modes (fewer, larger splits of
#endif                               // single requests: 0.3-1 us per layer less at batch 1)
#ifndef DSA_TUNE_MAX_FUSED_SPLIT
#define DSA_TUNE_MAX_FUSED_SPLIT 512  // most rows of a sparse-mode split (the fused step keeps
                                      // their logits and positions in LDS), vector-ALU tile
#endif
#ifndef DSA_TUNE_MAX_FUSED_SPLIT_MFMA
#define DSA_TUNE_MAX_FUSED_SPLIT_MFMA 512  // the same for the MFMA tile
#endif
#ifndef DSA_TUNE_UNROLL
#define DSA_TUNE_UNROLL 0  // loads in flight per wave (2, 4 or 8); 0: by group size
#endif
#ifndef DSA_TUNE_UNROLL_FP8
#define DSA_TUNE_UNROLL_FP8 5  // loads in flight per wave and operand on fp8 caches, at most
#endif                         // (d = 128: 40-row tiles, eight per Janus-like request, two per
                               // wave: 55.5 us per layer against 56.8 us with 6 and 57.8 us
                               // with 7; 8 spills registers)
#ifndef DSA_TUNE_VALU_WAVES
#define DSA_TUNE_VALU_WAVES 4  // most waves per workgroup of the vector-ALU decode tile
#endif
#ifndef DSA_TUNE_MFMA_WAVES
#define DSA_TUNE_MFMA_WAVES 8  // most waves per workgroup of the grouped-head MFMA tile
#endif
#ifndef DSA_TUNE_MFMA_WAVES_DENSE
#define DSA_TUNE_MFMA_WAVES_DENSE 2  // the same in dense mode (long rows, many workgroups)
#endif
#ifndef DSA_TUNE_KEPT_READ_PAIRS
#define DSA_TUNE_KEPT_READ_PAIRS 64  // selection states keep kept lists for the fused step in
#endif                               // launches of at most this many (request, KV head) pairs ...
#ifndef DSA_TUNE_KEPT_READ_CAP
#define DSA_TUNE_KEPT_READ_CAP 512   // ... or with skip lists longer than this (ranking exposed or
#endif                               // long; measured: large launches with short lists lose
                                     // 0.3-1 us per layer to the list stores)
#ifndef DSA_TUNE_VALU_GQA
#define DSA_TUNE_VALU_GQA 0  // 1: grouped query heads on the vector-ALU tile instead of MFMA
#endif

constexpr int kWaves = 4;          // waves per workgroup (the MFMA decode tile: kWavesMfma)
constexpr int kBlock = 64 * kWaves;
constexpr int kWavesMfma = DSA_TUNE_MFMA_WAVES;
constexpr int kWavesValu = DSA_TUNE_VALU_WAVES;
constexpr int kWavesMfmaDense = DSA_TUNE_MFMA_WAVES_DENSE;
static_assert(kWavesValu >= 1 && kWavesValu <= kWaves, "vector-ALU workgroup waves");
static_assert(kWavesMfma >= 1 && kWavesMfma <= 16, "MFMA workgroup waves");
static_assert(kWavesMfmaDense >= 1 && kWavesMfmaDense <= kWavesMfma, "MFMA workgroup waves");
constexpr int kMfmaTile = 32;        // rows per wave tile of the MFMA (grouped-head) path
constexpr int kMaxFusedSplit = DSA_TUNE_MAX_FUSED_SPLIT;
constexpr int kMaxFusedSplitMfma = DSA_TUNE_MAX_FUSED_SPLIT_MFMA;
constexpr int kSplitKbSparse = DSA_TUNE_SPLIT_KB;
constexpr int kSplitKbSparseMfma = DSA_TUNE_SPLIT_KB_MFMA;
constexpr int kSplitKbDense64 = DSA_TUNE_SPLIT_KB_DENSE_64;
constexpr int kSplitKbDense128 = DSA_TUNE_SPLIT_KB_DENSE_128;
constexpr int kSplitKbDenseMfma = DSA_TUNE_SPLIT_KB_DENSE_MFMA;
constexpr int kMinWorkgroups = DSA_TUNE_MIN_WGS;
constexpr int kMinWorkgroupsSparse = DSA_TUNE_MIN_WGS_SPARSE;
constexpr int kKeptReadPairs = DSA_TUNE_KEPT_READ_PAIRS;
constexpr int kKeptReadCap = DSA_TUNE_KEPT_READ_CAP;
// Longest kept list the fused step reads (the first 256 offsets are loaded
// ahead of the position): in launches of few pairs, and in the others.
constexpr int kKeptReadMax = 512;
constexpr int kKeptReadMaxWide = 256;
static_assert(kMaxFusedSplit % 64 == 0 && kMaxFusedSplit <= 1024, "fused split rows");
static_assert(kMaxFusedSplitMfma % 64 == 0 && kMaxFusedSplitMfma <= 1024, "fused split rows");
// Rows of one sparse-mode split at most, by tile.
constexpr int max_fused_split(bool mfma) { return mfma ? kMaxFusedSplitMfma : kMaxFusedSplit; }

// Grouped query heads take the MFMA tile (q.K^T and P.V on matrix cores).
constexpr bool uses_mfma_tile(int G) { return G >= 2 && !DSA_TUNE_VALU_GQA; }
// Loads in flight per wave and operand on the vector-ALU tile.
constexpr int unroll_of(int G) {
  return (DSA_TUNE_UNROLL == 2 || DSA_TUNE_UNROLL == 4 || DSA_TUNE_UNROLL == 8)
             ? DSA_TUNE_UNROLL
             : (G >= 8 ? 2 : (G >= 4 ? 4 : 8));
}
// The same for a cache of `elem_bytes`-byte elements and head_dim d: a tile
// holds at most 64 rows (one kept position per lane), and fp8 caches may be
// capped lower.  A lane loads 16 bytes, so one instruction covers
// 1024 / (d * elem_bytes) rows.
constexpr int unroll_for(int G, int d, int elem_bytes) {
  const int rpi = 1024 / (d * elem_bytes);
  int u = unroll_of(G);
  if (rpi * u > 64) u = 64 / rpi;
  if (elem_bytes == 1 && u > DSA_TUNE_UNROLL_FP8) u = DSA_TUNE_UNROLL_FP8;
  return u;
}
constexpr int kMaxFusedWindow = 16384;  // N_r of the fused step (skip bitmap per wave in LDS)
constexpr float kNegBig = -1.0e30f;  // "no score yet": finite, so exp2 of a difference is 0

struct PlanArgs {
  const int32_t* pos;
  const int32_t* st_count;
  const uint16_t* st_off;
  int32_t* count;
  int32_t* flags;
  int32_t* idx;
  int pairs, Hkv, Ldec, Nr, Natt, Ns, mode, plan_cap, state_cap, words;
};

struct DecodeArgs {
  const uint16_t* q;
  const uint8_t* k;      // K/V caches, addressed in bytes
  const uint8_t* v;
  const int64_t* row_base;  // per-request base offsets in elements, or nullptr
  int64_t sb, sh, sr;       // strides in bytes
  const float* ks;          // fp8: per-(request, KV head) K / V scales, or nullptr
  const float* vs;
  int kv_dtype;             // DSA_KV_BF16 or DSA_KV_FP8_E4M3
  const int32_t* pos;
  const int32_t* count;  // plan counts (diagonal mode)
  const int32_t* idx;    // plan indices (diagonal mode)
  float scale;           // sm_scale
  float scale_log2;      // sm_scale * log2(e)
  float* out;
  float* wlog;           // window logits or nullptr
  float* part;           // split partials (S > 1)
  int B, Hq, Hkv, Lp, Ldec, mode, plan_cap, C, S;
  int ring;              // positions >= Ns rotate through this many slots (0: linear)
  int Ns;                // sink positions
  // fused step only: selection state (in/out) and plan (out)
  int32_t* st_count;
  int32_t* st_flags;
  uint16_t* st_off;
  int32_t* plan_count;
  int32_t* plan_flags;
  int32_t* plan_idx;
  int32_t* st_kc;      // kept lists: tags [pairs][2] (k + 1, or 0) and lists (fused step)
  uint16_t* st_kept;
  int Nr, Natt, state_cap, words, kept_cap;
  int kept_read;       // 1: kept lists are stored by the selection and read by the fused step
};

struct SelectArgs {
  const int32_t* pos;
  const int32_t* count;  // plan counts
  const int32_t* idx;    // plan indices
  const float* wlog;
  int32_t* st_count;
  int32_t* st_flags;
  uint16_t* st_off;
  int32_t* st_kc;      // kept lists: tags [pairs][2] (k + 1, or 0) and lists
  uint16_t* st_kept;
  int pairs, Hq, Hkv, G, Ldec, Nr, Natt, Ns, plan_cap, state_cap, kept_cap, kept_stride;
  int kept_on;         // 1: the state's kept lists are kept (the fused step's launch rule)
};

struct ResetArgs {
  int32_t* st_count;
  int32_t* st_flags;
  int32_t* st_kc;
  const int32_t* mask;
  int pairs, Hkv;
};

hipError_t launch_plan(const Derived& d, const PlanArgs& a, hipStream_t st);
hipError_t launch_decode(const Derived& d, const DecodeArgs& a, hipStream_t st,
                         hipEvent_t t0 = nullptr, hipEvent_t t1 = nullptr);
hipError_t launch_step(const Derived& d, const DecodeArgs& a, hipStream_t st,
                       hipEvent_t t0 = nullptr, hipEvent_t t1 = nullptr);
// The fp8 instantiations (their own translation unit); fused selects the step.
hipError_t launch_kv_fp8(const Derived& d, const DecodeArgs& a, hipStream_t st, hipEvent_t t0,
                         hipEvent_t t1, bool fused);
hipError_t launch_select(const Derived& d, const SelectArgs& a, hipStream_t st);
hipError_t launch_reset(const Derived& d, const ResetArgs& a, hipStream_t st);

}  // namespace dsa

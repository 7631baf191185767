// Host side of the C ABI: argument validation, buffer layouts, the split
// configuration of the decode kernel, and the extern "C" entry points.
#include <cmath>
#include <mutex>

#include "internal.h"

namespace dsa {
namespace {

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

}  // namespace

dsa_status derive(const dsa_params* p, const dsa_shape* s, Derived* d) {
  if (!p || !s || !d) return DSA_ERR_INVALID_ARG;
  if (p->prompt_len < 0 || p->grid_h < 1 || p->grid_w < 1) return DSA_ERR_INVALID_ARG;
  if (p->mode != DSA_MODE_DENSE && p->mode != DSA_MODE_DIAGONAL && p->mode != DSA_MODE_WINDOW)
    return DSA_ERR_INVALID_ARG;
  if (p->window < 1 || p->window > 65535) return DSA_ERR_INVALID_ARG;
  // Window mode's recent window is N_att - S, not bounded by N_r.
  if (p->n_att < 1 || p->n_att > (p->mode == DSA_MODE_WINDOW ? (1 << 24) : p->window))
    return DSA_ERR_INVALID_ARG;
  if (p->sinks < 0 || (p->mode != DSA_MODE_DENSE && p->sinks >= p->n_att))
    return DSA_ERR_INVALID_ARG;
  const int64_t ldec = static_cast<int64_t>(p->grid_h) * p->grid_w;
  if (ldec > (1 << 24) || p->prompt_len > (1 << 24)) return DSA_ERR_INVALID_ARG;
  if (s->batch < 1 || s->num_q_heads < 1 || s->num_kv_heads < 1) return DSA_ERR_INVALID_ARG;
  if (s->num_q_heads % s->num_kv_heads) return DSA_ERR_INVALID_ARG;
  if (s->head_dim != 64 && s->head_dim != 128) return DSA_ERR_UNSUPPORTED;
  const int G = s->num_q_heads / s->num_kv_heads;
  if (G != 1 && G != 2 && G != 4 && G != 8) return DSA_ERR_UNSUPPORTED;
  const int64_t pairs = static_cast<int64_t>(s->batch) * s->num_kv_heads;
  if (pairs * s->num_q_heads / s->num_kv_heads * s->head_dim > (int64_t(1) << 31))
    return DSA_ERR_INVALID_ARG;

  d->B = s->batch;
  d->Hq = s->num_q_heads;
  d->Hkv = s->num_kv_heads;
  d->G = G;
  d->D = s->head_dim;
  d->Lp = p->prompt_len;
  d->Ldec = static_cast<int>(ldec);
  d->Natt = p->n_att;
  d->mode = p->mode;
  const bool sparse = p->mode != DSA_MODE_DENSE;  // a plan of kept rows (diagonal or window mode)
  d->Ns = sparse ? p->sinks : 0;
  d->Nr = p->mode == DSA_MODE_WINDOW ? p->n_att - p->sinks : p->window;
  d->plan_cap = sparse ? static_cast<int>(std::min<int64_t>(p->n_att, ldec)) : 0;
  d->state_cap = p->mode == DSA_MODE_DIAGONAL ? p->window - (p->n_att - p->sinks) : 0;
  d->words = d->state_cap > 0 ? (d->Nr + 31) / 32 : 0;
  if (pairs * std::max(d->plan_cap, 1) > (int64_t(1) << 30)) return DSA_ERR_INVALID_ARG;
  if (pairs * std::max(d->state_cap, 1) > (int64_t(1) << 30)) return DSA_ERR_INVALID_ARG;
  // Where it pays, every selection stores the kept list of the next step and
  // the fused step reads its kept rows from it instead of rebuilding them
  // from the skip entries: launches of few (request, KV head) pairs, whose
  // time is latency, and long skip lists (build-time constants, internal.h).
  // Elsewhere the lists are neither written nor read.
  {
    const int kept_cap = d->state_cap > 0 ? p->n_att - p->sinks : 0;
    const bool few = pairs <= kKeptReadPairs && kept_cap <= kKeptReadMax;
    const bool longs = d->state_cap > kKeptReadCap && kept_cap <= kKeptReadMaxWide;
    d->kept_read = kept_cap > 0 && (few || longs) ? 1 : 0;
  }

  // plan buffer: count | flags | indices
  size_t off = 0;
  d->plan.count_offset = off;
  off = align_up(off + 4 * pairs, 256);
  d->plan.flags_offset = off;
  off = align_up(off + 4 * pairs, 256);
  d->plan.indices_offset = off;
  off = align_up(off + 4 * static_cast<size_t>(pairs) * d->plan_cap, 256);
  d->plan.cap = d->plan_cap;
  d->plan.bytes = off;

  // state buffer: count | flags | offsets (uint16) | kept_count | kept (uint16)
  off = 0;
  d->state.count_offset = off;
  off = align_up(off + 4 * pairs, 256);
  d->state.flags_offset = off;
  off = align_up(off + 4 * pairs, 256);
  d->state.offsets_offset = off;
  off = align_up(off + 2 * static_cast<size_t>(pairs) * d->state_cap, 256);
  d->state.cap = d->state_cap;
  d->state.kept_cap = d->state_cap > 0 ? p->n_att - p->sinks : 0;
  // even, so every list starts on a 4-byte boundary
  d->state.kept_stride = (d->state.kept_cap + 1) & ~1;
  d->state.kept_count_offset = off;
  off = align_up(off + 4 * 2 * pairs, 256);
  d->state.kept_offset = off;
  off = align_up(off + 2 * 2 * static_cast<size_t>(pairs) * d->state.kept_stride, 256);
  d->state.bytes = off;

  // Split configuration of the decode kernel.  A wave issues U loads of
  // 512/d rows each (one tile) before consuming them; a split holds C rows
  // (a multiple of the tile), so every request is cut into a few workgroups
  // and the grid keeps enough loads in flight.  Every choice below is a
  // build-time constant (internal.h), so the launch shape and the workspace
  // size depend on the parameters and the shape alone.
  const int rows_per_instr = 512 / d->D;  // 8 for d=64, 4 for d=128
  d->MF = uses_mfma_tile(G);
  d->U = unroll_of(G);
  const int block_rows = d->MF ? kMfmaTile : rows_per_instr * d->U;
  const int64_t rows_max = d->Lp + (sparse ? d->plan_cap : ldec);
  d->rows_max = static_cast<int>(rows_max);
  // Measured on MI355X: dense splits of ~24 KB for d = 64 (long ragged rows
  // balance better), ~96 KB for d = 128 and ~128 KB for the grouped-head
  // tile (on two waves, several workgroups per CU).  Sparse-mode splits of
  // ~192 KB on the vector-ALU tile, so a Janus-like request (256 prompt
  // rows and 29 kept ones) is one split: no partials, no combine kernel,
  // and the selection stays in the decode kernel (8% faster per layer than
  // two splits, and faster on nearly every cell of the Janus-shaped sweep
  // with 16 or more requests).  ~256 KB on the MFMA tile, whose eight waves
  // keep two tiles each in flight: an Emu3-like request (256 prompt rows
  // and 205 kept ones) is one split too (16.0 us per layer against 24.1 us
  // with three splits and a combine).  The fused step caps a split at
  // max_fused_split rows.
  const int dense_kb = d->MF ? kSplitKbDenseMfma : (d->D == 64 ? kSplitKbDense64 : kSplitKbDense128);
  const int sparse_kb = d->MF ? kSplitKbSparseMfma : kSplitKbSparse;
  const int64_t split_bytes = (sparse ? sparse_kb : dense_kb) * int64_t(1024);
  int64_t c_target = std::max<int64_t>(block_rows, split_bytes / (4 * d->D));
  if (sparse) c_target = std::min<int64_t>(c_target, max_fused_split(d->MF));
  int64_t S = std::max<int64_t>(1, (rows_max + c_target - 1) / c_target);
  const int64_t min_wgs = sparse ? kMinWorkgroupsSparse : kMinWorkgroups;
  if (pairs * S < min_wgs) {
    const int64_t want = (min_wgs + pairs - 1) / pairs;
    const int64_t most = std::max<int64_t>(1, (rows_max + block_rows - 1) / block_rows);
    S = std::max<int64_t>(S, std::min(want, most));
  }
  int64_t C = (rows_max + S - 1) / S;
  C = std::max<int64_t>(block_rows, (C + block_rows - 1) / block_rows * block_rows);
  S = std::max<int64_t>(1, (rows_max + C - 1) / C);
  if (pairs * S > (int64_t(1) << 31) - 1) return DSA_ERR_INVALID_ARG;
  d->C = static_cast<int>(C);
  d->S = static_cast<int>(S);
  // Waves per workgroup: the most tiles any split has (tiles stop at the
  // prompt/decode boundary, so a split can have one more than C / tile).
  // fp8 caches load twice the elements per lane, so the vector-ALU tile
  // holds twice the rows (at most 64) and a split has fewer tiles.
  auto waves_for = [&](int64_t tile_rows) {
    int64_t max_tiles = 1;
    for (int64_t sp = 0; sp < S; ++sp) {
      const int64_t r0 = sp * C, r1 = std::min(rows_max, r0 + C);
      const int64_t pe = std::min<int64_t>(r1, d->Lp);
      const int64_t wst = std::max<int64_t>(r0, d->Lp);
      const int64_t tiles = (pe > r0 ? (pe - r0 + tile_rows - 1) / tile_rows : 0) +
                            (r1 > wst ? (r1 - wst + tile_rows - 1) / tile_rows : 0);
      max_tiles = std::max(max_tiles, tiles);
    }
    const int cap = d->MF ? (sparse ? kWavesMfma : kWavesMfmaDense) : kWavesValu;
    return static_cast<int>(std::min<int64_t>(cap, max_tiles));
  };
  d->NW = waves_for(block_rows);
  d->NW_fp8 = waves_for(d->MF ? kMfmaTile : 2 * rows_per_instr * unroll_for(G, d->D, 1));
  d->ws_bytes = S > 1 ? static_cast<size_t>(pairs) * S * G * (d->D + 2) * sizeof(float) : 0;
  return DSA_OK;
}

}  // namespace dsa

using dsa::Derived;

extern "C" {

DSA_API int32_t dsa_abi_version(void) { return DSA_ABI_VERSION; }

DSA_API const char* dsa_status_str(dsa_status st) {
  switch (st) {
    case DSA_OK: return "ok";
    case DSA_ERR_INVALID_ARG: return "invalid argument";
    case DSA_ERR_UNSUPPORTED: return "unsupported head_dim or head group size";
    case DSA_ERR_WORKSPACE: return "caller buffer too small";
    case DSA_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

DSA_API dsa_status dsa_params_from_sparsity(int32_t prompt_len, int32_t grid_h, int32_t grid_w,
                                            int32_t window, int32_t sparsity_permille,
                                            int32_t mode, int32_t sinks, dsa_params* out) {
  if (!out || sparsity_permille < 0 || sparsity_permille > 1000) return DSA_ERR_INVALID_ARG;
  if (prompt_len < 0 || grid_h < 1 || grid_w < 1 || window < 0 || window > 65535)
    return DSA_ERR_INVALID_ARG;
  if (mode != DSA_MODE_DENSE && mode != DSA_MODE_DIAGONAL && mode != DSA_MODE_WINDOW)
    return DSA_ERR_INVALID_ARG;
  const int64_t ldec = static_cast<int64_t>(grid_h) * grid_w;
  if (ldec > (1 << 24) || sinks < 0) return DSA_ERR_INVALID_ARG;
  int64_t nr = window;
  if (nr == 0) nr = std::max<int64_t>(1, std::min<int64_t>(ldec / 2, 65535));
  // round((1 - s) * L_dec) with ties up: floor((2 * (1000 - s) * L_dec + 1000) / 2000)
  int64_t natt = (2 * (1000 - int64_t(sparsity_permille)) * ldec + 1000) / 2000;
  natt = std::max<int64_t>(natt, int64_t(sinks) + 1);
  if (mode != DSA_MODE_WINDOW) natt = std::min(nr, natt);
  if (mode == DSA_MODE_DIAGONAL && sinks >= natt) return DSA_ERR_INVALID_ARG;
  out->prompt_len = prompt_len;
  out->grid_h = grid_h;
  out->grid_w = grid_w;
  out->window = static_cast<int32_t>(nr);
  out->n_att = static_cast<int32_t>(natt);
  out->mode = mode;
  out->sinks = sinks;
  return DSA_OK;
}

DSA_API dsa_status dsa_validate(const dsa_params* p, const dsa_shape* s) {
  Derived d;
  return dsa::derive(p, s, &d);
}

DSA_API dsa_status dsa_get_state_layout(const dsa_params* p, const dsa_shape* s,
                                        dsa_state_layout* out) {
  Derived d;
  dsa_status st = dsa::derive(p, s, &d);
  if (st != DSA_OK) return st;
  if (!out) return DSA_ERR_INVALID_ARG;
  *out = d.state;
  return DSA_OK;
}

DSA_API dsa_status dsa_get_plan_layout(const dsa_params* p, const dsa_shape* s,
                                       dsa_plan_layout* out) {
  Derived d;
  dsa_status st = dsa::derive(p, s, &d);
  if (st != DSA_OK) return st;
  if (!out) return DSA_ERR_INVALID_ARG;
  *out = d.plan;
  return DSA_OK;
}

DSA_API dsa_status dsa_get_launch_info(const dsa_params* p, const dsa_shape* s,
                                       dsa_launch_info* out) {
  Derived d;
  dsa_status st = dsa::derive(p, s, &d);
  if (st != DSA_OK) return st;
  if (!out) return DSA_ERR_INVALID_ARG;
  out->rows_per_split = d.C;
  out->max_splits = d.S;
  out->workgroups = d.B * d.Hkv * d.S;
  out->kernel_variant = d.MF ? 100 : d.U;
  out->waves_per_group = d.NW;
  out->workspace_bytes = d.ws_bytes;
  out->kept_read = d.kept_read;
  return DSA_OK;
}

DSA_API size_t dsa_state_bytes(const dsa_params* p, const dsa_shape* s) {
  Derived d;
  return dsa::derive(p, s, &d) == DSA_OK ? d.state.bytes : 0;
}

DSA_API size_t dsa_plan_bytes(const dsa_params* p, const dsa_shape* s) {
  Derived d;
  return dsa::derive(p, s, &d) == DSA_OK ? d.plan.bytes : 0;
}

DSA_API size_t dsa_workspace_bytes(const dsa_params* p, const dsa_shape* s) {
  Derived d;
  return dsa::derive(p, s, &d) == DSA_OK ? d.ws_bytes : 0;
}

DSA_API size_t dsa_window_logits_count(const dsa_params* p, const dsa_shape* s) {
  Derived d;
  return dsa::derive(p, s, &d) == DSA_OK
             ? static_cast<size_t>(d.B) * d.Hq * d.plan_cap
             : 0;
}

static dsa_status hip_status(hipError_t launch) {
  if (launch != hipSuccess) return DSA_ERR_HIP;
  return hipGetLastError() == hipSuccess ? DSA_OK : DSA_ERR_HIP;
}

DSA_API dsa_status dsa_state_reset(const dsa_params* p, const dsa_shape* s, void* d_state,
                                   const int32_t* d_req_mask, hipStream_t stream) {
  Derived d;
  dsa_status st = dsa::derive(p, s, &d);
  if (st != DSA_OK) return st;
  if (!d_state) return DSA_ERR_INVALID_ARG;
  char* base = static_cast<char*>(d_state);
  dsa::ResetArgs a{};
  a.st_count = reinterpret_cast<int32_t*>(base + d.state.count_offset);
  a.st_flags = reinterpret_cast<int32_t*>(base + d.state.flags_offset);
  a.st_kc = reinterpret_cast<int32_t*>(base + d.state.kept_count_offset);
  a.mask = d_req_mask;
  a.pairs = d.B * d.Hkv;
  a.Hkv = d.Hkv;
  return hip_status(dsa::launch_reset(d, a, stream));
}

DSA_API dsa_status dsa_plan(const dsa_params* p, const dsa_shape* s, const int32_t* d_decode_pos,
                            const void* d_state, void* d_plan, size_t plan_bytes,
                            hipStream_t stream) {
  Derived d;
  dsa_status st = dsa::derive(p, s, &d);
  if (st != DSA_OK) return st;
  if (!d_decode_pos || !d_plan) return DSA_ERR_INVALID_ARG;
  if (d.state_cap > 0 && !d_state) return DSA_ERR_INVALID_ARG;
  if (plan_bytes < d.plan.bytes) return DSA_ERR_WORKSPACE;
  char* pb = static_cast<char*>(d_plan);
  const char* sb = static_cast<const char*>(d_state);
  dsa::PlanArgs a{};
  a.pos = d_decode_pos;
  const bool has_state = sb && d.state_cap > 0;
  a.st_count = has_state ? reinterpret_cast<const int32_t*>(sb + d.state.count_offset) : nullptr;
  a.st_off = has_state ? reinterpret_cast<const uint16_t*>(sb + d.state.offsets_offset) : nullptr;
  a.count = reinterpret_cast<int32_t*>(pb + d.plan.count_offset);
  a.flags = reinterpret_cast<int32_t*>(pb + d.plan.flags_offset);
  a.idx = reinterpret_cast<int32_t*>(pb + d.plan.indices_offset);
  a.pairs = d.B * d.Hkv;
  a.Hkv = d.Hkv;
  a.Ldec = d.Ldec;
  a.Nr = d.Nr;
  a.Natt = d.Natt;
  a.Ns = d.Ns;
  a.mode = d.mode;
  a.plan_cap = d.plan_cap;
  a.state_cap = d.state_cap;
  a.words = d.words;
  return hip_status(dsa::launch_plan(d, a, stream));
}

// Shared by dsa_decode_attention (fused = false: reads the plan) and
// dsa_decode_step (fused = true: reads and updates the selection state and
// writes the plan).
static dsa_status decode_impl(const dsa_params* p, const dsa_shape* s, const void* d_q,
                              const void* d_k, const void* d_v, const dsa_kv_layout* kv,
                              const int32_t* d_decode_pos, const void* d_plan, float sm_scale,
                              float* d_out, float* d_window_logits, void* d_ws, size_t ws_bytes,
                              hipEvent_t t0, hipEvent_t t1, hipStream_t stream,
                              bool fused = false, void* d_state = nullptr,
                              size_t plan_bytes = 0) {
  Derived d;
  dsa_status st = dsa::derive(p, s, &d);
  if (st != DSA_OK) return st;
  if (!d_q || !d_k || !d_v || !kv || !d_decode_pos || !d_out) return DSA_ERR_INVALID_ARG;
  const bool sparse = d.mode != DSA_MODE_DENSE;
  if (sparse && !d_plan) return DSA_ERR_INVALID_ARG;
  if (fused && sparse) {
    if (d.state_cap > 0 && (!d_state || !d_window_logits)) return DSA_ERR_INVALID_ARG;
    if (plan_bytes < d.plan.bytes) return DSA_ERR_WORKSPACE;
    if (d.state_cap > 0 && d.Nr > dsa::kMaxFusedWindow) return DSA_ERR_UNSUPPORTED;
  }
  if (!std::isfinite(sm_scale)) return DSA_ERR_INVALID_ARG;
  if (kv->dtype != DSA_KV_BF16 && kv->dtype != DSA_KV_FP8_E4M3) return DSA_ERR_INVALID_ARG;
  if (kv->dtype == DSA_KV_BF16 && (kv->d_k_scale || kv->d_v_scale)) return DSA_ERR_INVALID_ARG;
  const int64_t esz = kv->dtype == DSA_KV_BF16 ? 2 : 1;
  if (kv->stride_row < d.D || kv->stride_head < 0 || kv->stride_batch < 0)
    return DSA_ERR_INVALID_ARG;
  if ((kv->stride_row | kv->stride_head | kv->stride_batch) & 7) return DSA_ERR_INVALID_ARG;
  if (kv->ring_rows < 0 || kv->ring_rows > (int64_t(1) << 30)) return DSA_ERR_INVALID_ARG;
  // The ring must hold every row a step can read: the sinks plus the window
  // (sparse modes), or every decode row (dense mode).
  if (kv->ring_rows > 0 &&
      kv->ring_rows < (sparse ? int64_t(d.Ns) + d.Nr : int64_t(d.Ldec)))
    return DSA_ERR_INVALID_ARG;
  if ((reinterpret_cast<uintptr_t>(d_k) | reinterpret_cast<uintptr_t>(d_v) |
       reinterpret_cast<uintptr_t>(d_q)) & 15)
    return DSA_ERR_INVALID_ARG;
  if (d.ws_bytes && (!d_ws || ws_bytes < d.ws_bytes)) return DSA_ERR_WORKSPACE;
  const char* pb = static_cast<const char*>(d_plan);
  dsa::DecodeArgs a{};
  a.q = static_cast<const uint16_t*>(d_q);
  a.k = static_cast<const uint8_t*>(d_k);
  a.v = static_cast<const uint8_t*>(d_v);
  a.row_base = kv->d_row_base;
  a.sb = kv->stride_batch * esz;
  a.sh = kv->stride_head * esz;
  a.sr = kv->stride_row * esz;
  a.ks = kv->d_k_scale;
  a.vs = kv->d_v_scale;
  a.kv_dtype = kv->dtype;
  a.pos = d_decode_pos;
  a.count = pb ? reinterpret_cast<const int32_t*>(pb + d.plan.count_offset) : nullptr;
  a.idx = pb ? reinterpret_cast<const int32_t*>(pb + d.plan.indices_offset) : nullptr;
  a.scale = sm_scale;
  a.scale_log2 = sm_scale * 1.4426950408889634f;
  a.out = d_out;
  a.wlog = sparse ? d_window_logits : nullptr;
  a.part = static_cast<float*>(d_ws);
  a.B = d.B;
  a.Hq = d.Hq;
  a.Hkv = d.Hkv;
  a.Lp = d.Lp;
  a.Ldec = d.Ldec;
  a.mode = d.mode;
  a.plan_cap = d.plan_cap;
  a.C = d.C;
  a.S = d.S;
  // No ring (0), or a ring of at least L_dec slots, maps every position to
  // itself; otherwise a.ring >= N_r > 0 slots rotate after the sinks.
  a.ring = (kv->ring_rows == 0 || kv->ring_rows >= d.Ldec)
               ? 0
               : static_cast<int>(kv->ring_rows - d.Ns);
  a.Ns = d.Ns;
  a.Nr = d.Nr;
  a.Natt = d.Natt;
  a.state_cap = d.state_cap;
  a.words = d.words;
  if (fused && sparse) {
    char* sb = static_cast<char*>(d_state);
    char* pbw = static_cast<char*>(const_cast<void*>(d_plan));
    if (d.state_cap > 0) {
      a.st_count = reinterpret_cast<int32_t*>(sb + d.state.count_offset);
      a.st_flags = reinterpret_cast<int32_t*>(sb + d.state.flags_offset);
      a.st_off = reinterpret_cast<uint16_t*>(sb + d.state.offsets_offset);
      a.st_kc = reinterpret_cast<int32_t*>(sb + d.state.kept_count_offset);
      a.st_kept = reinterpret_cast<uint16_t*>(sb + d.state.kept_offset);
      a.kept_cap = d.state.kept_cap;
      a.kept_read = d.kept_read;
    }
    a.plan_count = reinterpret_cast<int32_t*>(pbw + d.plan.count_offset);
    a.plan_flags = reinterpret_cast<int32_t*>(pbw + d.plan.flags_offset);
    a.plan_idx = reinterpret_cast<int32_t*>(pbw + d.plan.indices_offset);
    a.count = nullptr;
    a.idx = nullptr;
    return hip_status(dsa::launch_step(d, a, stream, t0, t1));
  }
  return hip_status(dsa::launch_decode(d, a, stream, t0, t1));
}

DSA_API dsa_status dsa_decode_attention(const dsa_params* p, const dsa_shape* s, const void* d_q,
                                        const void* d_k, const void* d_v,
                                        const dsa_kv_layout* kv, const int32_t* d_decode_pos,
                                        const void* d_plan, float sm_scale, float* d_out,
                                        float* d_window_logits, void* d_ws, size_t ws_bytes,
                                        hipStream_t stream) {
  return decode_impl(p, s, d_q, d_k, d_v, kv, d_decode_pos, d_plan, sm_scale, d_out,
                     d_window_logits, d_ws, ws_bytes, nullptr, nullptr, stream);
}

DSA_API dsa_status dsa_decode_attention_timed(const dsa_params* p, const dsa_shape* s,
                                              const void* d_q, const void* d_k, const void* d_v,
                                              const dsa_kv_layout* kv,
                                              const int32_t* d_decode_pos, const void* d_plan,
                                              float sm_scale, float* d_out,
                                              float* d_window_logits, void* d_ws, size_t ws_bytes,
                                              hipEvent_t decode_start, hipEvent_t decode_stop,
                                              hipStream_t stream) {
  if (!decode_start || !decode_stop) return DSA_ERR_INVALID_ARG;
  return decode_impl(p, s, d_q, d_k, d_v, kv, d_decode_pos, d_plan, sm_scale, d_out,
                     d_window_logits, d_ws, ws_bytes, decode_start, decode_stop, stream);
}

DSA_API dsa_status dsa_decode_step(const dsa_params* p, const dsa_shape* s, const void* d_q,
                                   const void* d_k, const void* d_v, const dsa_kv_layout* kv,
                                   const int32_t* d_decode_pos, void* d_state, void* d_plan,
                                   size_t plan_bytes, float sm_scale, float* d_out,
                                   float* d_window_logits, void* d_ws, size_t ws_bytes,
                                   hipStream_t stream) {
  return decode_impl(p, s, d_q, d_k, d_v, kv, d_decode_pos, d_plan, sm_scale, d_out,
                     d_window_logits, d_ws, ws_bytes, nullptr, nullptr, stream, true, d_state,
                     plan_bytes);
}

DSA_API dsa_status dsa_decode_step_timed(const dsa_params* p, const dsa_shape* s, const void* d_q,
                                         const void* d_k, const void* d_v,
                                         const dsa_kv_layout* kv, const int32_t* d_decode_pos,
                                         void* d_state, void* d_plan, size_t plan_bytes,
                                         float sm_scale, float* d_out, float* d_window_logits,
                                         void* d_ws, size_t ws_bytes, hipEvent_t decode_start,
                                         hipEvent_t decode_stop, hipStream_t stream) {
  if (!decode_start || !decode_stop) return DSA_ERR_INVALID_ARG;
  return decode_impl(p, s, d_q, d_k, d_v, kv, d_decode_pos, d_plan, sm_scale, d_out,
                     d_window_logits, d_ws, ws_bytes, decode_start, decode_stop, stream, true,
                     d_state, plan_bytes);
}

}  // extern "C"

// Split partials of dsa_decode_step_noalloc: a file-scope device array, one
// copy per GPU, held until the process ends.  Host code never passes the
// array's name to a kernel (on the host it is only a stand-in for the
// symbol); it uses the device address hipGetSymbolAddress returns on each
// GPU, looked up once per device on the first call made with that device
// current.  Nothing needs clearing between calls: each split writes its own
// partial before the combine reads it, and the combine reads only splits
// that exist.
static __device__ __align__(256) unsigned char scratch[DSA_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's copy of `scratch`, or nullptr.
void* scratch_on_current_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return nullptr;
    g_scratch_ptr[dev] = ptr;
  }
  return g_scratch_ptr[dev];
}

}  // namespace

extern "C" {

DSA_API dsa_status dsa_decode_step_noalloc(const dsa_params* p, const dsa_shape* s,
                                           const void* d_q, const void* d_k, const void* d_v,
                                           const dsa_kv_layout* kv, const int32_t* d_decode_pos,
                                           void* d_state, void* d_plan, size_t plan_bytes,
                                           float sm_scale, float* d_out, float* d_window_logits,
                                           hipStream_t stream) {
  Derived d;
  dsa_status st = dsa::derive(p, s, &d);
  if (st != DSA_OK) return st;
  if (d.ws_bytes > DSA_NOALLOC_SCRATCH_BYTES) return DSA_ERR_WORKSPACE;
  void* ws = nullptr;
  if (d.ws_bytes) {
    ws = scratch_on_current_device();
    if (!ws) return DSA_ERR_HIP;
  }
  return decode_impl(p, s, d_q, d_k, d_v, kv, d_decode_pos, d_plan, sm_scale, d_out,
                     d_window_logits, ws, d.ws_bytes ? DSA_NOALLOC_SCRATCH_BYTES : 0, nullptr,
                     nullptr, stream, true, d_state, plan_bytes);
}

DSA_API dsa_status dsa_select(const dsa_params* p, const dsa_shape* s, const int32_t* d_decode_pos,
                              const void* d_plan, const float* d_window_logits, void* d_state,
                              hipStream_t stream) {
  Derived d;
  dsa_status st = dsa::derive(p, s, &d);
  if (st != DSA_OK) return st;
  // Dense and window mode keep no selection; nor does N_att - S == N_r.
  if (d.state_cap == 0) return DSA_OK;
  if (!d_decode_pos || !d_plan || !d_window_logits || !d_state) return DSA_ERR_INVALID_ARG;
  const char* pb = static_cast<const char*>(d_plan);
  char* sb = static_cast<char*>(d_state);
  dsa::SelectArgs a{};
  a.pos = d_decode_pos;
  a.count = reinterpret_cast<const int32_t*>(pb + d.plan.count_offset);
  a.idx = reinterpret_cast<const int32_t*>(pb + d.plan.indices_offset);
  a.wlog = d_window_logits;
  a.st_count = reinterpret_cast<int32_t*>(sb + d.state.count_offset);
  a.st_flags = reinterpret_cast<int32_t*>(sb + d.state.flags_offset);
  a.st_off = reinterpret_cast<uint16_t*>(sb + d.state.offsets_offset);
  a.st_kc = reinterpret_cast<int32_t*>(sb + d.state.kept_count_offset);
  a.st_kept = reinterpret_cast<uint16_t*>(sb + d.state.kept_offset);
  a.kept_cap = d.state.kept_cap;
  a.kept_stride = d.state.kept_stride;
  a.kept_on = d.kept_read;
  a.pairs = d.B * d.Hkv;
  a.Hq = d.Hq;
  a.Hkv = d.Hkv;
  a.G = d.G;
  a.Ldec = d.Ldec;
  a.Nr = d.Nr;
  a.Natt = d.Natt;
  a.Ns = d.Ns;
  a.plan_cap = d.plan_cap;
  a.state_cap = d.state_cap;
  return hip_status(dsa::launch_select(d, a, stream));
}

}  // extern "C"

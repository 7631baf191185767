/*
 * dsa.h -- diagonal-aware sparse decode attention on AMD Instinct MI355X
 * (gfx950): the C ABI of libdsa.so.
 *
 * The library computes the decode-phase attention of an autoregressive
 * image generator with the kept-KV selection of Algorithm 1 of the paper
 * (section 4, "Diagonal-Aware Sparse Attention"):
 *
 *   - every step's keys include all L_p prompt rows;
 *   - inside a recent window of N_r decode positions, a per-head list of
 *     skipped entries grows by one per step during phase 2 (an argmin of the
 *     window softmax) and then stays fixed; because both the list entries and
 *     the step index advance by +1 per step, every entry is stored as its
 *     relative offset d = t - j, which never changes, so the per-step "shift"
 *     of the algorithm costs nothing;
 *   - each step attends exactly min(t + 1, N_att) decode rows;
 *   - the variants of section 5.1 keep the first S decode tokens as
 *     attention sinks ("Diagonal+Sink4": Algorithm 1 on the later tokens;
 *     StreamingLLM: the sinks plus a recent window; S = 0 is the plain
 *     sliding window);
 *   - a dense mode (all decode rows 0 .. t) is the baseline the paper
 *     compares against in its evaluation (section 5).
 *
 * A decode step for one layer is:
 *
 *     dsa_plan              kept decode positions per (request, KV head)
 *     dsa_decode_attention  split-K attention over prompt + kept rows, then
 *                           the cross-split log-sum-exp combine
 *     dsa_select            phase-2 argmin, appends one offset per KV head
 *
 * Conventions for every call:
 *   - Pointers named d_* are DEVICE pointers owned by the caller.  The
 *     library never allocates device memory and keeps no device state between
 *     calls; buffer sizes come from the *_bytes queries.  (The one exception
 *     is dsa_decode_step_noalloc, whose split partials live in a fixed
 *     per-GPU buffer inside the library.)
 *   - Calls that take a hipStream_t only enqueue work on that stream and
 *     return without synchronising; results are visible to later work on the
 *     same stream.  Calls on distinct buffers may run concurrently.
 *   - Every entry point returns a dsa_status; no C++ exception crosses the
 *     ABI.  Arguments are validated on the host before anything is enqueued.
 *   - Device-side precondition failures (a decode position outside the grid,
 *     a corrupt selection state) never cause an out-of-bounds access: the
 *     value is clamped or ignored and a bit is set in the per-(request, KV
 *     head) flag words of the plan or state buffer.
 *   - Query head h reads KV head h / (num_q_heads / num_kv_heads).
 *   - "bf16" is IEEE bfloat16; "fp32" is IEEE binary32.
 */
#ifndef DSA_H_
#define DSA_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DSA_API __attribute__((visibility("default")))

#define DSA_ABI_VERSION 4

/* ---- status codes -------------------------------------------------------- */
typedef int32_t dsa_status;
#define DSA_OK               0
#define DSA_ERR_INVALID_ARG (-1) /* a NULL pointer or an out-of-range value */
#define DSA_ERR_UNSUPPORTED (-2) /* valid but not built: head_dim, group size */
#define DSA_ERR_WORKSPACE   (-3) /* a caller buffer is smaller than required */
#define DSA_ERR_HIP         (-4) /* the HIP runtime refused a launch */

/* ---- modes ----------------------------------------------------------------- */
#define DSA_MODE_DENSE    0 /* attend prompt + decode rows 0 .. t            */
#define DSA_MODE_DIAGONAL 1 /* attend prompt + the rows Algorithm 1 keeps     */
#define DSA_MODE_WINDOW   2 /* attend prompt + sinks + the most recent rows   */

/* ---- KV cache element types ------------------------------------------------ */
#define DSA_KV_BF16     0 /* IEEE bfloat16                                     */
#define DSA_KV_FP8_E4M3 1 /* OCP 8-bit float E4M3 ("FN": no infinities,
                             max 448) times a per-(request, KV head) scale  */

/* ---- per-(request, KV head) flag bits (plan and state buffers) ------------ */
#define DSA_FLAG_INACTIVE      1  /* decode position < 0: request slot unused   */
#define DSA_FLAG_POS_CLAMPED   2  /* decode position >= H*W, clamped to H*W-1   */
#define DSA_FLAG_STATE_BEHIND  4  /* fewer skip entries than the step needs     */
#define DSA_FLAG_BAD_OFFSET    8  /* a stored offset outside [0, N_r-2] ignored */
#define DSA_FLAG_COUNT         16 /* kept count differs from min(t+1, N_att)    */

/*
 * Method parameters (Algorithm 1 inputs, section 4; sinks, section 5.1).
 *   prompt_len  L_p >= 0, prompt rows always attended
 *   grid_h/w    visual token grid, >= 1; L_dec = grid_h * grid_w decode steps
 *   window      N_r, recent window, 1 <= N_r <= 65535 (checked in every
 *               mode, used by DSA_MODE_DIAGONAL only)
 *   n_att       N_att, decode rows attended per step, including the sinks;
 *               1 <= N_att, and N_att <= N_r in DSA_MODE_DIAGONAL
 *   mode        DSA_MODE_DENSE, DSA_MODE_DIAGONAL or DSA_MODE_WINDOW
 *   sinks       S, 0 <= S < N_att: decode positions 0 .. S-1 are always
 *               attended once decoded.  DSA_MODE_DIAGONAL runs Algorithm 1
 *               on the positions after them as if position S were step 0
 *               (window N_r, N_att - S rows to attend: "Diagonal+Sink4" is
 *               S = 4); DSA_MODE_WINDOW attends the sinks plus the
 *               N_att - S most recent positions (StreamingLLM is S = 4, the
 *               sliding window S = 0).  Ignored in dense mode.
 * In every sparse mode a step attends min(t + 1, N_att) decode rows.
 */
typedef struct dsa_params {
  int32_t prompt_len;
  int32_t grid_h;
  int32_t grid_w;
  int32_t window;
  int32_t n_att;
  int32_t mode;
  int32_t sinks;
} dsa_params;

/*
 * Problem shape of one layer.
 *   batch        B >= 1 requests
 *   num_q_heads  Hq >= 1
 *   num_kv_heads Hkv >= 1, Hq % Hkv == 0, group Hq / Hkv in {1, 2, 4, 8}
 *   head_dim     d in {64, 128}
 */
typedef struct dsa_shape {
  int32_t batch;
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t head_dim;
} dsa_shape;

/*
 * Where row r of KV head h of request b lives in the K and V arrays (both
 * arrays share one layout and one element type).  Rows 0 .. L_p-1 are the
 * prompt.  Element offset of a row's first element:
 *     base(b) + h * stride_head + r * stride_row
 * with base(b) = d_row_base[b] when d_row_base is non-NULL (a device array of
 * B int64 values, e.g. for ragged packing), else b * stride_batch.
 * Decode position j is row L_p + j (ring_rows = 0, a linear cache), or,
 * when ring_rows = R > 0, a ring: the S sink positions keep rows
 * L_p .. L_p + S - 1 (S = 0 in dense mode) and position j >= S lives in row
 * L_p + S + ((j - S) mod (R - S)), overwriting position j - (R - S).  In
 * diagonal mode this is the physical form of Algorithm 1's eviction (phase 3
 * drops K[t - N_r], so per section 4, "Cost analysis", no more than
 * L_p + N_r rows of a head are ever live) and needs R >= S + N_r; window
 * mode needs R >= N_att; dense mode reads every decode row, so a ring must
 * hold R >= H*W there.  A ring of R >= H*W rows is the linear cache.
 * A row holds head_dim contiguous elements of type dtype:
 *   DSA_KV_BF16      2 bytes each; d_k_scale and d_v_scale must be NULL.
 *   DSA_KV_FP8_E4M3  1 byte each; element value = E4M3 value of the byte
 *                    times d_k_scale[b*Hkv + h] (K) or d_v_scale[b*Hkv + h]
 *                    (V), fp32 device arrays of B*Hkv scales, or 1 where the
 *                    pointer is NULL.  Bytes 0x7F and 0xFF (NaN) give
 *                    unspecified outputs.  KV quantization is orthogonal to
 *                    the selection (section 6): it halves the bytes per kept
 *                    key and changes nothing else.
 * The K/V base pointers must be 16-byte aligned, and every base(b),
 * stride_head and stride_row must be a multiple of 8 elements.  The caller
 * guarantees every row the step reads exists and holds the KV of the
 * position it stands for (linear: rows up to L_p + t_b; ring: the sinks and
 * the slots of the positions the step can keep).
 */
typedef struct dsa_kv_layout {
  const int64_t* d_row_base;
  int64_t stride_batch;
  int64_t stride_head;
  int64_t stride_row;
  int64_t ring_rows;
  const float* d_k_scale;
  const float* d_v_scale;
  int32_t dtype;
} dsa_kv_layout;

/* Byte offsets of the arrays inside a plan buffer (all int32):
 *   count  [B*Hkv]           kept decode rows of (b, h), index b*Hkv + h
 *   flags  [B*Hkv]           DSA_FLAG_* bits
 *   indices[B*Hkv][cap]      kept decode positions of (b, h), ascending
 * cap = min(N_att, L_dec) in the sparse modes and 0 in dense mode.       */
typedef struct dsa_plan_layout {
  size_t count_offset;
  size_t flags_offset;
  size_t indices_offset;
  int32_t cap;
  size_t bytes;
} dsa_plan_layout;

/* Byte offsets of the arrays inside a selection-state buffer:
 *   count      int32  [B*Hkv]            skip entries stored for (b, h)
 *   flags      int32  [B*Hkv]            DSA_FLAG_* bits set by dsa_select
 *   offsets    uint16 [B*Hkv][cap]       skip entries as offsets d = t - j, in
 *                                        the order Algorithm 1 appends them
 *   kept_count int32  [B*Hkv][2]         slot s: k + 1 when list s below holds
 *                                        the window's kept offsets after the
 *                                        first k skip entries (k even in slot 0,
 *                                        odd in slot 1); 0 when it holds none
 *   kept       uint16 [B*Hkv][2][kept_stride]  the two lists: kept_cap
 *                                        offsets each, largest first (oldest
 *                                        position first)
 * cap = N_r - (N_att - S) in diagonal mode (the largest skip list of
 * Algorithm 1 over the positions after the S sinks), 0 in the other modes
 * (nothing is selected; the state buffer may then be NULL everywhere).
 * kept_cap = N_att - S in diagonal mode, else 0; kept_stride = kept_cap
 * rounded up to an even number.
 * After k skip entries the window holds the offsets 0 .. N_att - 1 - S + k
 * (at most N_r - 1), of which the k stored ones are skipped: N_att - S kept
 * offsets, a function of the stored entries alone.  Where the launch rule
 * turns them on (dsa_launch_info.kept_read), every phase-2 selection writes
 * the list for the next step into the other slot (the new oldest offset
 * leads, the selected one leaves), so the fused step reads its kept rows
 * instead of rebuilding them from the skip entries, and repeating a step
 * finds its list still there; a list that does not match the step
 * (kept_count != k + 1) is ignored and the kept rows are rebuilt.  A caller
 * that rewrites the skip entries itself sets kept_count to 0.  Zero-filled
 * memory and dsa_state_reset leave no list; with kept_read = 0 the two
 * sections are neither written nor read.                                  */
typedef struct dsa_state_layout {
  size_t count_offset;
  size_t flags_offset;
  size_t offsets_offset;
  int32_t cap;
  size_t bytes;
  size_t kept_count_offset;
  size_t kept_offset;
  int32_t kept_cap;
  int32_t kept_stride;
} dsa_state_layout;

/* How dsa_decode_attention splits the keys (for reports and tests).  The
 * split rule is fixed when the library is built: it depends on the
 * parameters and the shape of a call and on nothing else. */
typedef struct dsa_launch_info {
  int32_t rows_per_split;  /* C: keys per split workgroup                   */
  int32_t max_splits;      /* S: splits per (request, KV head) at most      */
  int32_t workgroups;      /* B * Hkv * S                                   */
  int32_t kernel_variant;  /* K/V loads in flight per wave (2, 4 or 8), or 100 for
                              the MFMA tile of grouped query heads (32 rows) */
  int32_t waves_per_group; /* waves per split workgroup (1..4; MFMA tile 1..8) */
  size_t workspace_bytes;  /* fp32 partials for the combine                 */
  int32_t kept_read;       /* 1: selections keep the state's kept lists and
                              dsa_decode_step reads its kept window rows from
                              them when they match; a function of (params,
                              shape): launches of at most 64 (request, KV
                              head) pairs with kept_cap <= 512, or with
                              cap > 512 and kept_cap <= 256                 */
} dsa_launch_info;

/* ---- host-only helpers (no device work) ---------------------------------- */

/* ABI version (DSA_ABI_VERSION of the built library). */
DSA_API int32_t dsa_abi_version(void);

/* Human-readable message for a status code; never NULL. */
DSA_API const char* dsa_status_str(dsa_status status);

/*
 * Fill *out from a target sparsity (section 5.1: sparsity = 1 - N_att/L_dec)
 * and the window rule of the "Parameter selection" paragraph of section 4.
 *   window = 0 selects the paper's default N_r = L_dec / 2 (at least 1);
 *   n_att = floor((1000 - sparsity_permille) * L_dec / 1000 + 1/2),
 *           computed in integers, then raised to at least sinks + 1 and, in
 *           dense and diagonal mode, lowered to at most N_r (window mode
 *           keeps it up to L_dec: its recent window is not bounded by N_r).
 * Errors: DSA_ERR_INVALID_ARG for out == NULL, sparsity outside [0, 1000],
 * negative prompt_len, grid < 1, window outside [0, 65535], a bad mode,
 * sinks < 0, or sinks >= N_r in diagonal mode.
 */
DSA_API dsa_status dsa_params_from_sparsity(int32_t prompt_len, int32_t grid_h, int32_t grid_w,
                                            int32_t window, int32_t sparsity_permille,
                                            int32_t mode, int32_t sinks, dsa_params* out);

/* Validate a parameter/shape pair as every device call does.  Returns
 * DSA_OK, DSA_ERR_INVALID_ARG or DSA_ERR_UNSUPPORTED. */
DSA_API dsa_status dsa_validate(const dsa_params* p, const dsa_shape* s);

/* Buffer layouts; *out is filled only on DSA_OK. */
DSA_API dsa_status dsa_get_state_layout(const dsa_params* p, const dsa_shape* s,
                                        dsa_state_layout* out);
DSA_API dsa_status dsa_get_plan_layout(const dsa_params* p, const dsa_shape* s,
                                       dsa_plan_layout* out);
DSA_API dsa_status dsa_get_launch_info(const dsa_params* p, const dsa_shape* s,
                                       dsa_launch_info* out);

/* Sizes in bytes (0 when p/s are invalid). */
DSA_API size_t dsa_state_bytes(const dsa_params* p, const dsa_shape* s);
DSA_API size_t dsa_plan_bytes(const dsa_params* p, const dsa_shape* s);
DSA_API size_t dsa_workspace_bytes(const dsa_params* p, const dsa_shape* s);
/* Number of fp32 window logits per call: B * Hq * cap (plan cap). */
DSA_API size_t dsa_window_logits_count(const dsa_params* p, const dsa_shape* s);

/* ---- device calls ---------------------------------------------------------- */

/*
 * Empty the skip lists of the selected requests: Algorithm 1 starts every
 * request with skip_idx = [].  Clears count and flags of (b, h) for every KV
 * head h of each request b with d_req_mask[b] != 0 (every request when
 * d_req_mask is NULL).  d_state: state buffer of dsa_state_bytes bytes.
 * Uses a kernel, never a memset, so it may be captured in a HIP graph.
 */
DSA_API dsa_status dsa_state_reset(const dsa_params* p, const dsa_shape* s, void* d_state,
                                   const int32_t* d_req_mask, hipStream_t stream);

/*
 * Kept decode positions of one step (Algorithm 1: "window - skip_idx" with
 * window = [max(0, t-N_r), .., t] and K[t-N_r] evicted in phase 3).
 *   d_decode_pos  int32 [B]: t_b, the newest decode position of request b
 *                 (its K/V row L_p + t_b is already written); t_b < 0 marks
 *                 an unused slot (count 0, output zeros).
 *   d_state       selection state; the step uses the first
 *                 clamp(t_b - N_att + 1, 0, state cap) entries of each list
 *                 (the entries appended at steps < t_b), so replaying a step
 *                 is exact.  Ignored (may be NULL) when the state cap is 0
 *                 (dense and window mode, or N_att - S = N_r).
 *   d_plan        output, plan_bytes >= dsa_plan_bytes().  For each (b, h):
 *                 count = kept rows (sparse modes: min(t_b+1, N_att)), flags,
 *                 and in the sparse modes the kept positions, ascending: the
 *                 sinks 0 .. min(S, t_b+1)-1, then t_b - d for the offsets
 *                 d in [0, min(t_b - S, W - 1)] not in the skip list, with
 *                 W = N_r (diagonal) or N_att - S (window).
 * Errors: INVALID_ARG (NULL pointers, bad params), UNSUPPORTED, WORKSPACE
 * (plan_bytes too small), HIP.
 */
DSA_API dsa_status dsa_plan(const dsa_params* p, const dsa_shape* s, const int32_t* d_decode_pos,
                            const void* d_state, void* d_plan, size_t plan_bytes,
                            hipStream_t stream);

/*
 * Attn(Q_t, K_p + K[idx], V_p + V[idx]) of Algorithm 1 for every request and
 * query head: softmax(sm_scale * q . k) over the prompt rows plus the kept
 * decode rows of the plan (diagonal mode) or all decode rows 0 .. t_b (dense
 * mode), times V.  Keys are split into chunks processed by independent
 * workgroups with an fp32 online softmax; a second kernel merges the chunks
 * by log-sum-exp when a request has more than one.
 *   d_q              bf16 [B][Hq][d]
 *   d_k, d_v         bf16 or fp8 caches in the dsa_kv_layout layout
 *   d_decode_pos     int32 [B] as for dsa_plan
 *   d_plan           plan of the same step (sparse modes); may be NULL in
 *                    dense mode
 *   sm_scale         softmax scale, normally 1/sqrt(d)
 *   d_out            fp32 [B][Hq][d]; zeros for unused slots
 *   d_window_logits  NULL, or fp32 [B][Hq][cap]: sm_scale * q . k of every
 *                    kept decode row in plan order, sinks included (sparse
 *                    modes; entries past count are not written; k is the
 *                    scaled value for fp8 caches).  dsa_select reads them.
 *   d_ws, ws_bytes   workspace of at least dsa_workspace_bytes() bytes
 * Errors: INVALID_ARG, UNSUPPORTED, WORKSPACE, HIP.
 */
DSA_API dsa_status dsa_decode_attention(const dsa_params* p, const dsa_shape* s, const void* d_q,
                                        const void* d_k, const void* d_v,
                                        const dsa_kv_layout* kv, const int32_t* d_decode_pos,
                                        const void* d_plan, float sm_scale, float* d_out,
                                        float* d_window_logits, void* d_ws, size_t ws_bytes,
                                        hipStream_t stream);

/*
 * dsa_decode_attention with its kernels launched so that decode_start
 * receives the split-K kernel's own start timestamp and decode_stop the end
 * timestamp of the last kernel of the call (the split-K kernel, or the
 * combine when a request is split), through the AMD extended launch;
 * hipEventElapsedTime(decode_start, decode_stop) is then the call's
 * execution time on the device, without the queueing ahead of it.  The
 * events must already exist (hipEventCreate).  For profiling tools; not
 * usable inside a HIP graph capture.  Errors as dsa_decode_attention, and
 * INVALID_ARG for a NULL event.
 */
DSA_API dsa_status dsa_decode_attention_timed(const dsa_params* p, const dsa_shape* s,
                                              const void* d_q, const void* d_k, const void* d_v,
                                              const dsa_kv_layout* kv,
                                              const int32_t* d_decode_pos, const void* d_plan,
                                              float sm_scale, float* d_out,
                                              float* d_window_logits, void* d_ws, size_t ws_bytes,
                                              hipEvent_t decode_start, hipEvent_t decode_stop,
                                              hipStream_t stream);

/*
 * One whole decode step of one layer in a single pass over the KV:
 * exactly dsa_plan -> dsa_decode_attention -> dsa_select (diagonal mode)
 * with bit-identical plan, window logits, output and selection state, the
 * way the paper's own kernel fuses the index gather and the window argmin
 * into the attention (section 5.1, "Implementation").  Every decode
 * workgroup rebuilds the kept set of its (request, KV head) from d_state,
 * or reads it from the state's kept list where the launch keeps them
 * (dsa_launch_info.kept_read); when one split covers a (request, KV head)
 * it also runs the phase-2
 * argmin and appends the skip entry, otherwise a second kernel merges the
 * splits and selects.  In dense mode it is dsa_decode_attention and d_state,
 * d_plan and d_window_logits are not used.
 *   d_state          selection state, in/out; may be NULL when the state
 *                    cap is 0 (window mode, or N_att - S = N_r)
 *   d_plan           plan of this step, out; plan_bytes >= dsa_plan_bytes()
 *   d_window_logits  fp32 [B][Hq][cap], out; required when the state cap is
 *                    not 0, else optional
 *   other arguments  as for dsa_decode_attention
 * Errors: as dsa_decode_attention; UNSUPPORTED for N_r > 16384 in diagonal
 * mode with a non-zero state cap (use the three separate calls there).
 */
DSA_API dsa_status dsa_decode_step(const dsa_params* p, const dsa_shape* s, const void* d_q,
                                   const void* d_k, const void* d_v, const dsa_kv_layout* kv,
                                   const int32_t* d_decode_pos, void* d_state, void* d_plan,
                                   size_t plan_bytes, float sm_scale, float* d_out,
                                   float* d_window_logits, void* d_ws, size_t ws_bytes,
                                   hipStream_t stream);

/* dsa_decode_step with the start of its split-K kernel and the end of its
 * last kernel recorded into two existing events (as
 * dsa_decode_attention_timed). */
DSA_API dsa_status dsa_decode_step_timed(const dsa_params* p, const dsa_shape* s, const void* d_q,
                                         const void* d_k, const void* d_v,
                                         const dsa_kv_layout* kv, const int32_t* d_decode_pos,
                                         void* d_state, void* d_plan, size_t plan_bytes,
                                         float sm_scale, float* d_out, float* d_window_logits,
                                         void* d_ws, size_t ws_bytes, hipEvent_t decode_start,
                                         hipEvent_t decode_stop, hipStream_t stream);

/*
 * dsa_decode_step for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same step with the same results, bit for bit, but without a workspace
 * argument.  The split partials go to a buffer of
 * DSA_NOALLOC_SCRATCH_BYTES bytes inside the library, one per GPU, held
 * until the process ends.  The call allocates nothing and needs no memset.
 *   arguments   as dsa_decode_step (the caller still passes the state, plan,
 *               window logits and output buffers)
 * Every call on one GPU shares that GPU's buffer: two calls on one GPU whose
 * execution overlaps (different streams, no ordering between them) race and
 * give undefined results; calls ordered on one stream are safe.
 * Errors: as dsa_decode_step; WORKSPACE when the call would need more
 * partials than the buffer holds (dsa_workspace_bytes() >
 * DSA_NOALLOC_SCRATCH_BYTES: use dsa_decode_step with a caller workspace);
 * HIP when the buffer's device address cannot be obtained.
 */
#define DSA_NOALLOC_SCRATCH_BYTES (16u << 20)
DSA_API dsa_status dsa_decode_step_noalloc(const dsa_params* p, const dsa_shape* s,
                                           const void* d_q, const void* d_k, const void* d_v,
                                           const dsa_kv_layout* kv, const int32_t* d_decode_pos,
                                           void* d_state, void* d_plan, size_t plan_bytes,
                                           float sm_scale, float* d_out, float* d_window_logits,
                                           hipStream_t stream);

/*
 * Phase-2 selection of Algorithm 1: for every request with
 * N_att - 1 <= t_b <= N_r + S - 2 and every KV head h, compute
 *   w_q = softmax(window logits of query head q)   over the kept window
 *                                                  (the sinks excluded)
 *   sigma_j = sum of w_q[j] over the query heads q that read KV head h
 *   j* = argmin_j sigma_j (first, i.e. oldest, on ties)
 * and store offset t_b - idx[j*] as skip entry number k = t_b - N_att + 1
 * (count becomes k + 1).  At group size 1 the argmin is taken on the logits,
 * which orders exactly as the softmax.  Requests outside that step range,
 * and the modes without a selection state, are left untouched.  A state
 * with fewer than k entries is left unchanged and flagged
 * DSA_FLAG_STATE_BEHIND.
 *   d_plan, d_window_logits  from dsa_plan / dsa_decode_attention of this step
 *   d_state                  in/out
 * Errors: INVALID_ARG, UNSUPPORTED, HIP.
 */
DSA_API dsa_status dsa_select(const dsa_params* p, const dsa_shape* s, const int32_t* d_decode_pos,
                              const void* d_plan, const float* d_window_logits, void* d_state,
                              hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* DSA_H_ */

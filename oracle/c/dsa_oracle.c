/*
 * CPU oracle in plain C (fp64): Algorithm 1 of the paper (section 4) for one
 * head, and one decode step of one request over all its KV heads.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path links or calls
 * this file: only the tests, the smoke check and the CPU-baseline leg of the
 * benchmark do.  It shares no code, header or table with the HIP library.
 * It restates the same definitions as the Python oracle (oracle/alg1.py,
 * oracle/attention.py, oracle/step.py) so that long selection histories
 * (windows of thousands of positions) and whole requests can be computed in
 * seconds; the tests pin it to the Python oracle and to the paper's worked
 * example.
 *
 * Algorithm 1, as stored here: skip_idx is a list of absolute decode
 * positions; at the start of every step of phase 2 or 3 each entry moves one
 * position along its diagonal (+1); in phase 3 (t >= N_r) position t - N_r
 * leaves the cache (evicted[] marks it); the step attends the window
 * [max(0, t - N_r), t] minus the evicted and the skipped positions; a phase-2
 * step (N_att - 1 <= t < N_r) with fewer than N_r - N_att entries then
 * appends one more position, chosen by the caller or by the argmin of the
 * window softmax.  The appended entry is still attended at its own step.
 *
 * Attention: out_h = sum_j softmax_j(scale * q_h . k_j) v_j over the prompt
 * rows followed by the kept decode rows, with the maximum subtracted before
 * exponentiation.  Selection score of window key j for a KV head: the sum
 * over the group's query heads of softmax(scale * q_h . k_j) taken over the
 * kept window keys only; the first (oldest) minimum wins.
 *
 * Build: gcc -O2 -fopenmp -shared -fPIC (no fast-math: IEEE fp64).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_API __attribute__((visibility("default")))

enum { ORC_OK = 0, ORC_ERR_ARG = -1, ORC_ERR_RAND = -2, ORC_ERR_MEM = -3 };

/* Phase of step t: 1 before the first selection, 2 while the window grows,
 * 3 once it slides. */
static int phase_of(int N_r, int N_att, int t) {
  if (t < N_att - 1) return 1;
  return t < N_r ? 2 : 3;
}

/*
 * One step of Algorithm 1 for one head.
 *   skip[0 .. *n_skip)  skip_idx, absolute positions (capacity N_r - N_att)
 *   evicted[0 .. L)     1 for positions whose KV has left the cache
 *   mark[0 .. L + 1)    caller scratch, all zero on entry and on return
 * Writes the kept positions (ascending) to idx / *n_idx and whether this
 * step adds a skip entry to *adds; the caller appends with orc_append.
 * Returns ORC_ERR_ARG when t is outside [0, L).
 */
static int alg1_step(int N_r, int N_att, int t, int L, int32_t* skip, int32_t* n_skip,
                     uint8_t* evicted, uint8_t* mark, int32_t* idx, int32_t* n_idx, int* adds) {
  if (t < 0 || t >= L) return ORC_ERR_ARG;
  const int ph = phase_of(N_r, N_att, t);
  *adds = ph == 2 && *n_skip < N_r - N_att;
  if (ph == 3) evicted[t - N_r] = 1;
  if (ph >= 2)
    for (int i = 0; i < *n_skip; ++i) skip[i] += 1;
  for (int i = 0; i < *n_skip; ++i)
    if (skip[i] >= 0 && skip[i] <= L) mark[skip[i]] = 1;
  int n = 0;
  const int lo = t - N_r > 0 ? t - N_r : 0;
  for (int j = lo; j <= t; ++j)
    if (!evicted[j] && !mark[j]) idx[n++] = j;
  for (int i = 0; i < *n_skip; ++i)
    if (skip[i] >= 0 && skip[i] <= L) mark[skip[i]] = 0;
  *n_idx = n;
  return ORC_OK;
}

/*
 * Selection states after steps 0 .. t_end - 1 of one head, each choice being
 * rand[k] mod |idx| for the k-th selecting step, followed by step t_end
 * itself (no choice made at it): its kept positions go to idx / *n_idx and
 * the skip list it used stays in skip / *n_skip.  evicted must hold L zero
 * bytes on entry, skip room for N_r - N_att entries, idx room for N_r + 1.
 * Returns ORC_OK, ORC_ERR_ARG, ORC_ERR_RAND (too few random values) or
 * ORC_ERR_MEM.
 */
ORC_API int orc_alg1_replay(int32_t N_r, int32_t N_att, int32_t L, int32_t t_end,
                            const int64_t* rand, int64_t n_rand, int32_t* skip, int32_t* n_skip,
                            uint8_t* evicted, int32_t* idx, int32_t* n_idx) {
  if (N_att < 1 || N_att > N_r || t_end < 0 || t_end >= L) return ORC_ERR_ARG;
  uint8_t* mark = (uint8_t*)calloc((size_t)L + 2, 1);
  if (!mark) return ORC_ERR_MEM;
  *n_skip = 0;
  int64_t k = 0;
  int st = ORC_OK;
  for (int t = 0; t <= t_end && st == ORC_OK; ++t) {
    int adds = 0;
    st = alg1_step(N_r, N_att, t, L, skip, n_skip, evicted, mark, idx, n_idx, &adds);
    if (st != ORC_OK || t == t_end || !adds) continue;
    if (k >= n_rand || *n_idx < 1) {
      st = ORC_ERR_RAND;
      break;
    }
    const int64_t r = rand[k++];
    const int j = (int)(((r % *n_idx) + *n_idx) % *n_idx);
    skip[(*n_skip)++] = idx[j];
  }
  free(mark);
  return st;
}

/* Single-query attention of one query head over nk key rows given as row
 * pointers, fp64. */
static void attend(int d, int nk, const double* q, const double* const* krow,
                   const double* const* vrow, double scale, double* s, double* out) {
  double mx = -INFINITY;
  for (int j = 0; j < nk; ++j) {
    double acc = 0.0;
    for (int i = 0; i < d; ++i) acc += q[i] * krow[j][i];
    s[j] = scale * acc;
    if (s[j] > mx) mx = s[j];
  }
  double z = 0.0;
  for (int i = 0; i < d; ++i) out[i] = 0.0;
  for (int j = 0; j < nk; ++j) {
    const double w = exp(s[j] - mx);
    z += w;
    for (int i = 0; i < d; ++i) out[i] += w * vrow[j][i];
  }
  for (int i = 0; i < d; ++i) out[i] /= z;
}

/*
 * One decode step t of one request, every KV head, fp64:
 *   dims = {Hq, Hkv, d, L_p, N_r, N_att, L, mode (0 dense, 1 diagonal)}
 *   q        [Hq][d]
 *   Kp, Vp   [Hkv][L_p][d]
 *   K, V     [Hkv][rows][d]: decode position j is row j (rows > t)
 *   skip     [Hkv][N_r - N_att], n_skip [Hkv], evicted [Hkv][L]: the
 *            per-KV-head Algorithm 1 states, updated in place (diagonal)
 *   out      [Hq][d]
 *   picked   [Hkv]: the position appended at this step, or -1
 *   threads  OpenMP threads over the KV heads (>= 1)
 * Query head h reads KV head h / (Hq / Hkv).  Returns ORC_OK, ORC_ERR_ARG
 * or ORC_ERR_MEM.
 */
ORC_API int orc_request_step(const int32_t* dims, int32_t t, const double* q, const double* Kp,
                             const double* Vp, const double* K, const double* V, int32_t rows,
                             double scale, int32_t* skip, int32_t* n_skip, uint8_t* evicted,
                             double* out, int32_t* picked, int32_t threads) {
  const int Hq = dims[0], Hkv = dims[1], d = dims[2], Lp = dims[3], N_r = dims[4],
            N_att = dims[5], L = dims[6], mode = dims[7];
  if (Hq < 1 || Hkv < 1 || Hq % Hkv || d < 1 || Lp < 0 || t < 0 || t >= L || rows <= t ||
      threads < 1 || (mode != 0 && mode != 1) || (mode == 1 && (N_att < 1 || N_att > N_r)))
    return ORC_ERR_ARG;
  const int g = Hq / Hkv;
  const int cap = mode == 1 ? N_r - N_att : 0;
  int status = ORC_OK;
#pragma omp parallel for num_threads(threads) schedule(dynamic, 1)
  for (int h = 0; h < Hkv; ++h) {
    const int nmax = Lp + t + 1;
    int32_t* idx = (int32_t*)malloc(sizeof(int32_t) * (size_t)(t + 1));
    const double** kr = (const double**)malloc(sizeof(double*) * (size_t)nmax);
    const double** vr = (const double**)malloc(sizeof(double*) * (size_t)nmax);
    double* s = (double*)malloc(sizeof(double) * (size_t)nmax);
    double* sigma = (double*)malloc(sizeof(double) * (size_t)(t + 1));
    uint8_t* mark = (uint8_t*)calloc((size_t)L + 2, 1);
    if (!idx || !kr || !vr || !s || !sigma || !mark) {
#pragma omp atomic write
      status = ORC_ERR_MEM;
    } else {
      int n = 0, adds = 0;
      if (mode == 0) {
        for (int j = 0; j <= t; ++j) idx[n++] = j;
      } else {
        alg1_step(N_r, N_att, t, L, skip + (size_t)h * cap, n_skip + h, evicted + (size_t)h * L,
                  mark, idx, &n, &adds);
      }
      for (int j = 0; j < Lp; ++j) {
        kr[j] = Kp + ((size_t)h * Lp + j) * d;
        vr[j] = Vp + ((size_t)h * Lp + j) * d;
      }
      for (int j = 0; j < n; ++j) {
        kr[Lp + j] = K + ((size_t)h * rows + idx[j]) * d;
        vr[Lp + j] = V + ((size_t)h * rows + idx[j]) * d;
      }
      for (int i = 0; i < n; ++i) sigma[i] = 0.0;
      for (int gi = 0; gi < g; ++gi) {
        const double* qh = q + (size_t)(h * g + gi) * d;
        attend(d, Lp + n, qh, kr, vr, scale, s, out + (size_t)(h * g + gi) * d);
        if (adds) {
          /* window softmax over the kept decode keys (s[Lp ..] are their
             scaled logits) */
          double mx = -INFINITY, z = 0.0;
          for (int j = 0; j < n; ++j)
            if (s[Lp + j] > mx) mx = s[Lp + j];
          for (int j = 0; j < n; ++j) z += exp(s[Lp + j] - mx);
          for (int j = 0; j < n; ++j) sigma[j] += exp(s[Lp + j] - mx) / z;
        }
      }
      picked[h] = -1;
      if (adds && n > 0) {
        int jb = 0;
        for (int j = 1; j < n; ++j)
          if (sigma[j] < sigma[jb]) jb = j;
        skip[(size_t)h * cap + n_skip[h]] = idx[jb];
        n_skip[h] += 1;
        picked[h] = idx[jb];
      }
    }
    free(idx);
    free(kr);
    free(vr);
    free(s);
    free(sigma);
    free(mark);
  }
  return status;
}

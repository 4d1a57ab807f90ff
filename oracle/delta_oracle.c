/*
 * delta_oracle.c -- plain fp64 CPU oracle of the Delta Attention prefill.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may link, load or
 * call this file: only the tests, the smoke check and the benchmark's CPU
 * baseline leg use it.  It shares no code, header, table or helper with the
 * GPU library.
 *
 * What it computes (Delta Attention: Fast and Accurate Sparse Attention
 * Inference by Delta Correction, arXiv 2505.11254):
 *
 *   f  : dense causal softmax attention, scale 1/sqrt(d), keys j <= i
 *        (Sec. 2, Eq. "attention"; causality: row i sees keys j <= i).
 *   f* : StreamingLLM sparse attention -- sink tokens plus a sliding window,
 *        softmax normalised over the selected keys only (Sec. 1-2 and the
 *        normalisation remark before Lemma 1 in Sec. 3).
 *        S(i) = { j <= i : j < n_sink  or  i - j < window }.
 *   Algorithm 1 (Sec. 3):
 *     1. A*V  <- f*(Q,K,V)                 for every row
 *     2. Q~   <- every gamma-th row of Q   (Eq. "q-index-selection")
 *     3. A~V  <- f(Q~,K,V)
 *     4. Delta <- A~V - (A*V)_{i in delta}, delta = { i : i mod gamma = 0 }
 *     5. out  <- A*V + repeat(Delta, gamma)   (Eq. "delta-final")
 *   Implementation-details appendix: the last rows that do not fill a whole
 *   group of gamma rows are computed densely, so the corrected part has a
 *   length divisible by gamma.
 *
 * Readings taken where the paper is silent or garbled:
 *   - positions are 0-based and local to each sequence; anchors are the rows
 *     i with i mod gamma = 0, row i uses the anchor floor(i/gamma)*gamma <= i;
 *   - the window holds `window` keys including the query itself (i - j < w);
 *   - sinks are the first n_sink positions, united with the window;
 *   - scale 1/sqrt(d) for both f and f* (Eq. 4 omits it; Eq. 1 has it);
 *   - GQA: query head h reads kv head floor(h / (Hq/Hkv));
 *   - tail rows [L_c, L), L_c = floor(L/gamma)*gamma, take the dense result.
 *
 * Arithmetic: every score, exponential, normaliser and output is fp64.
 * Inputs are either fp64 or IEEE bfloat16 bit patterns, which are widened
 * to fp64 exactly (a bfloat16 is the top half of a binary32).
 * Softmax is two-pass per row: scores and their max, then exp(x - max),
 * the normaliser Z and the weighted value sum.
 *
 * Layout: token-major contiguous tensors, q/out [T, Hq, d], k/v [T, Hkv, d];
 * sequence b occupies rows [cu[b], cu[b+1]).
 *
 * Other sparse bases (the method corrects any sparse attention f*: Sec. 3,
 * and the MInference/HiP/Star-Attention comparisons of Sec. 4): f* given by
 * key-block lists.  Keys are grouped in tiles of 64 positions and query rows
 * in blocks of block_q rows (positions local to the sequence).  For sequence
 * b, kv head g and query block qb, the list holds the key tiles that the
 * block's rows attend to; the tiles overlapping the query block itself
 * (tile >= qb*block_q/64) are always attended; listed entries outside
 * [0, qb*block_q/64) are ignored.  Row i then sees
 *   S(i) = { j <= i : tile(j) listed for (b, kv(h), i / block_q) or
 *                     tile(j) >= (i / block_q) * block_q / 64 },
 * normalised over S(i) only, and Algorithm 1 runs unchanged on top.
 * Lists are CSR: ptr [B][Hkv][nqb + 1] offsets into idx.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define DAO_OK 0
#define DAO_ERR_ARG 1
#define DAO_ERR_NOMEM 2

#define DAO_MODE_DENSE 0
#define DAO_MODE_SPARSE 1
#define DAO_MODE_BLOCKS 2 /* f* from key-block lists */
#define DAO_TILE 64       /* keys per tile of the block lists */

typedef struct {
  const void* q;
  const void* k;
  const void* v;
  int in_bf16; /* 1: inputs are bfloat16 bit patterns, 0: fp64 */
  const int64_t* cu; /* host, B + 1 entries */
  int B, Hq, Hkv, d;
  int window, n_sink;
  /* key-block lists (DAO_MODE_BLOCKS only) */
  const int64_t* blk_ptr; /* [B][Hkv][nqb + 1] */
  const int64_t* blk_idx;
  int nqb, block_q;
} dao_problem;

/* Widen element idx of an input tensor to fp64 (exact for bfloat16). */
static inline double ld(const void* p, int bf16, int64_t idx) {
  if (bf16) {
    uint32_t u = ((uint32_t)((const uint16_t*)p)[idx]) << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
  }
  return ((const double*)p)[idx];
}

/*
 * Selected key tiles of row i under the block lists: sel[t] = 1 for every
 * tile t <= i / 64 in S(i).  sel needs i / 64 + 1 entries.
 */
static void block_row_tiles(const dao_problem* P, int b, int g, int64_t i, unsigned char* sel) {
  const int64_t qb = i / P->block_q;
  const int64_t diag0 = qb * P->block_q / DAO_TILE; /* first tile of the query block */
  const int64_t last = i / DAO_TILE;
  for (int64_t t = 0; t <= last; ++t) sel[t] = (t >= diag0);
  const int64_t* ptr = P->blk_ptr + ((int64_t)b * P->Hkv + g) * (P->nqb + 1);
  for (int64_t e = ptr[qb]; e < ptr[qb + 1]; ++e) {
    const int64_t t = P->blk_idx[e];
    if (t >= 0 && t < diag0) sel[t] = 1;
  }
}

/* Key j (<= i) belongs to the key set of row i under the given mode; for
 * DAO_MODE_BLOCKS, sel holds the row's selected tiles. */
static inline int key_in_set(int mode, int64_t i, int64_t j, int window, int n_sink,
                             const unsigned char* sel) {
  if (j > i) return 0;                 /* causal */
  if (mode == DAO_MODE_DENSE) return 1;
  if (mode == DAO_MODE_BLOCKS) return sel[j / DAO_TILE];
  return (j < n_sink) || (i - j < window);
}

/*
 * One attention row: query row i (local) of head h in sequence b, over the
 * key set of `mode`.  Writes o[d]; *m_out / *z_out receive the score max and
 * the normaliser sum_j exp(x_j - m) when non-NULL; w_out (length i+1), when
 * non-NULL, receives the softmax weight of every key j <= i (0 outside the
 * set).  `x` is scratch of at least i+1 doubles, followed (for the block
 * lists) by i/64 + 1 bytes of tile flags.
 */
static void attn_row(const dao_problem* P, int mode, int b, int h, int64_t i,
                     double* o, double* m_out, double* z_out, double* w_out, double* x) {
  const int d = P->d;
  const int G = P->Hq / P->Hkv;
  const int g = h / G;
  unsigned char* sel = (unsigned char*)(x + i + 1);
  if (mode == DAO_MODE_BLOCKS) block_row_tiles(P, b, g, i, sel);
  const int64_t base = P->cu[b];
  const double tau = 1.0 / sqrt((double)d);
  const int64_t qoff = ((base + i) * P->Hq + h) * (int64_t)d;

  /* pass 1: scores over the key set and their max */
  double m = -INFINITY;
  for (int64_t j = 0; j <= i; ++j) {
    if (!key_in_set(mode, i, j, P->window, P->n_sink, sel)) continue;
    const int64_t koff = ((base + j) * P->Hkv + g) * (int64_t)d;
    double s = 0.0;
#pragma omp simd reduction(+ : s)
    for (int c = 0; c < d; ++c) s += ld(P->q, P->in_bf16, qoff + c) * ld(P->k, P->in_bf16, koff + c);
    x[j] = tau * s;
    if (x[j] > m) m = x[j];
  }
  /* pass 2: exponentials, normaliser, weighted values */
  double z = 0.0;
  for (int c = 0; c < d; ++c) o[c] = 0.0;
  for (int64_t j = 0; j <= i; ++j) {
    if (!key_in_set(mode, i, j, P->window, P->n_sink, sel)) continue;
    const double p = exp(x[j] - m);
    z += p;
    const int64_t voff = ((base + j) * P->Hkv + g) * (int64_t)d;
#pragma omp simd
    for (int c = 0; c < d; ++c) o[c] += p * ld(P->v, P->in_bf16, voff + c);
  }
  for (int c = 0; c < d; ++c) o[c] /= z;
  if (m_out) *m_out = m;
  if (z_out) *z_out = z;
  if (w_out) {
    for (int64_t j = 0; j <= i; ++j)
      w_out[j] = key_in_set(mode, i, j, P->window, P->n_sink, sel) ? exp(x[j] - m) / z : 0.0;
  }
}

static int check_problem(const dao_problem* P) {
  if (!P->q || !P->k || !P->v || !P->cu) return DAO_ERR_ARG;
  if (P->B < 1 || P->Hq < 1 || P->Hkv < 1 || P->d < 1) return DAO_ERR_ARG;
  if (P->Hq % P->Hkv != 0) return DAO_ERR_ARG;
  if (P->window < 1 || P->n_sink < 0) return DAO_ERR_ARG;
  for (int b = 0; b < P->B; ++b)
    if (P->cu[b + 1] < P->cu[b]) return DAO_ERR_ARG;
  return DAO_OK;
}

static int64_t max_len(const dao_problem* P) {
  int64_t L = 0;
  for (int b = 0; b < P->B; ++b)
    if (P->cu[b + 1] - P->cu[b] > L) L = P->cu[b + 1] - P->cu[b];
  return L;
}

/*
 * Plain attention (f or f*) for every row, or for a list of rows.
 * rows == NULL: out is [T, Hq, d]; m_out / z_out (optional) are [T, Hq].
 * rows != NULL: n_rows triples (b, h, i_local); out is [n_rows, d];
 *               m_out / z_out (optional) are [n_rows].
 */
int dao_attention(const void* q, const void* k, const void* v, int in_bf16,
                  const int64_t* cu, int B, int Hq, int Hkv, int d,
                  int window, int n_sink, int mode,
                  const int64_t* rows, int64_t n_rows,
                  double* out, double* m_out, double* z_out, int nthreads) {
  dao_problem P = {q, k, v, in_bf16, cu, B, Hq, Hkv, d, window, n_sink, NULL, NULL, 0, 0};
  if (mode != DAO_MODE_DENSE && mode != DAO_MODE_SPARSE) return DAO_ERR_ARG;
  if (mode == DAO_MODE_DENSE) { P.window = 1; P.n_sink = 0; } /* unused by f */
  if (check_problem(&P) != DAO_OK || !out) return DAO_ERR_ARG;
  const int64_t T = cu[B];
  const int64_t Lmax = max_len(&P);
  int64_t n_items = rows ? n_rows : T * Hq;
  int err = DAO_OK;
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#else
  (void)nthreads;
#endif
#pragma omp parallel
  {
    double* x = (double*)malloc(sizeof(double) * (size_t)(Lmax + 1) + (size_t)(Lmax / DAO_TILE + 1));
    if (!x) {
#pragma omp atomic write
      err = DAO_ERR_NOMEM;
    }
#pragma omp for schedule(dynamic, 16)
    for (int64_t it = 0; it < n_items; ++it) {
      if (!x) continue;
      int b, h;
      int64_t i;
      double *o, *mo, *zo;
      if (rows) {
        b = (int)rows[3 * it];
        h = (int)rows[3 * it + 1];
        i = rows[3 * it + 2];
        o = out + it * d;
        mo = m_out ? m_out + it : NULL;
        zo = z_out ? z_out + it : NULL;
      } else {
        const int64_t t = it / Hq;
        h = (int)(it % Hq);
        b = 0;
        while (cu[b + 1] <= t) ++b;
        i = t - cu[b];
        o = out + it * d;
        mo = m_out ? m_out + it : NULL;
        zo = z_out ? z_out + it : NULL;
      }
      if (b < 0 || b >= B || h < 0 || h >= Hq || i < 0 || i >= cu[b + 1] - cu[b]) {
#pragma omp atomic write
        err = DAO_ERR_ARG;
        continue;
      }
      attn_row(&P, mode, b, h, i, o, mo, zo, NULL, x);
    }
    free(x);
  }
  return err;
}

/*
 * Softmax weights of one row (b, h, i) under `mode`: w[j] for j = 0..i, zero
 * outside the key set.  Used by the tests to check normalisation and support.
 */
int dao_attention_weights(const void* q, const void* k, const void* v, int in_bf16,
                          const int64_t* cu, int B, int Hq, int Hkv, int d,
                          int window, int n_sink, int mode, int b, int h, int64_t i,
                          double* w, double* o) {
  dao_problem P = {q, k, v, in_bf16, cu, B, Hq, Hkv, d, window, n_sink, NULL, NULL, 0, 0};
  if (mode != DAO_MODE_DENSE && mode != DAO_MODE_SPARSE) return DAO_ERR_ARG;
  if (mode == DAO_MODE_DENSE) { P.window = 1; P.n_sink = 0; } /* unused by f */
  if (check_problem(&P) != DAO_OK || !w || !o) return DAO_ERR_ARG;
  if (b < 0 || b >= B || h < 0 || h >= Hq || i < 0 || i >= cu[b + 1] - cu[b]) return DAO_ERR_ARG;
  double* x = (double*)malloc(sizeof(double) * (size_t)(i + 1) + (size_t)(i / DAO_TILE + 1));
  if (!x) return DAO_ERR_NOMEM;
  attn_row(&P, mode, b, h, i, o, NULL, NULL, w, x);
  free(x);
  return DAO_OK;
}

/*
 * Delta Attention, Algorithm 1, over whole sequences.
 *   out    [T, Hq, d]  the corrected output (required)
 *   sparse [T, Hq, d]  A*V for every row            (optional)
 *   delta  [T, Hq, d]  the correction added to each row (optional; zero on
 *                      tail rows, where the dense result replaces the row)
 */
static int delta_full(const dao_problem* Pp, int smode, int gamma, double* out,
                      double* sparse_out, double* delta_out, int nthreads) {
  const dao_problem P = *Pp;
  const int64_t* cu = P.cu;
  const int B = P.B, Hq = P.Hq, d = P.d;
  const int64_t T = cu[B];
  const int64_t Lmax = max_len(&P);
  double* sp = sparse_out ? sparse_out : (double*)malloc(sizeof(double) * (size_t)(T * Hq * d + 1));
  if (!sp) return DAO_ERR_NOMEM;
  int err = DAO_OK;
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#else
  (void)nthreads;
#endif
  /* Step 1: A*V <- f*(Q, K, V) for every row of every sequence and head. */
#pragma omp parallel
  {
    double* x = (double*)malloc(sizeof(double) * (size_t)(Lmax + 1) + (size_t)(Lmax / DAO_TILE + 1));
#pragma omp for schedule(dynamic, 16)
    for (int64_t it = 0; it < T * Hq; ++it) {
      if (!x) {
#pragma omp atomic write
        err = DAO_ERR_NOMEM;
        continue;
      }
      const int64_t t = it / Hq;
      const int h = (int)(it % Hq);
      int b = 0;
      while (cu[b + 1] <= t) ++b;
      attn_row(&P, smode, b, h, t - cu[b], sp + it * d, NULL, NULL, NULL, x);
    }
    free(x);
  }
  if (err != DAO_OK) { if (!sparse_out) free(sp); return err; }

  /* Steps 2-5, per sequence and head. */
#pragma omp parallel
  {
    double* x = (double*)malloc(sizeof(double) * (size_t)(Lmax + 1) + (size_t)(Lmax / DAO_TILE + 1));
    double* dense = (double*)malloc(sizeof(double) * (size_t)d);
    double* dl = (double*)malloc(sizeof(double) * (size_t)d);
#pragma omp for schedule(dynamic, 1) collapse(2)
    for (int b = 0; b < B; ++b) {
      for (int h = 0; h < Hq; ++h) {
        if (!x || !dense || !dl) {
#pragma omp atomic write
          err = DAO_ERR_NOMEM;
          continue;
        }
        const int64_t L = cu[b + 1] - cu[b];
        const int64_t Lc = (L / gamma) * gamma; /* corrected prefix */
        /* Steps 2-4: for every anchor a in delta = {0, gamma, ...} < Lc, the
         * dense row f(Q~_a) and Delta_a = A~V_a - (A*V)_a; step 5 adds Delta_a
         * to the gamma rows a .. a+gamma-1 (repeat(Delta, gamma)). */
        for (int64_t a = 0; a < Lc; a += gamma) {
          attn_row(&P, DAO_MODE_DENSE, b, h, a, dense, NULL, NULL, NULL, x);
          const double* spa = sp + ((cu[b] + a) * Hq + h) * (int64_t)d;
          for (int c = 0; c < d; ++c) dl[c] = dense[c] - spa[c];
          for (int64_t i = a; i < a + gamma; ++i) {
            const int64_t off = ((cu[b] + i) * Hq + h) * (int64_t)d;
            for (int c = 0; c < d; ++c) out[off + c] = sp[off + c] + dl[c];
            if (delta_out)
              for (int c = 0; c < d; ++c) delta_out[off + c] = dl[c];
          }
        }
        /* Tail rows [Lc, L): computed densely (implementation-details appendix). */
        for (int64_t i = Lc; i < L; ++i) {
          const int64_t off = ((cu[b] + i) * Hq + h) * (int64_t)d;
          attn_row(&P, DAO_MODE_DENSE, b, h, i, out + off, NULL, NULL, NULL, x);
          if (delta_out)
            for (int c = 0; c < d; ++c) delta_out[off + c] = 0.0;
        }
      }
    }
    free(x);
    free(dense);
    free(dl);
  }
  if (!sparse_out) free(sp);
  return err;
}

int dao_delta_attention(const void* q, const void* k, const void* v, int in_bf16,
                        const int64_t* cu, int B, int Hq, int Hkv, int d,
                        int window, int n_sink, int gamma,
                        double* out, double* sparse_out, double* delta_out, int nthreads) {
  dao_problem P = {q, k, v, in_bf16, cu, B, Hq, Hkv, d, window, n_sink, NULL, NULL, 0, 0};
  if (check_problem(&P) != DAO_OK || !out || gamma < 1) return DAO_ERR_ARG;
  return delta_full(&P, DAO_MODE_SPARSE, gamma, out, sparse_out, delta_out, nthreads);
}

/*
 * Delta Attention at selected rows only: for each (b, h, i) the value row i
 * of the full algorithm takes.  A row needs its own sparse key set and the
 * dense and sparse results of its anchor floor(i/gamma)*gamma, so any subset
 * is exact.  out is [n_rows, d]; delta (optional) is [n_rows, d].
 */
static int delta_rows(const dao_problem* Pp, int smode, int gamma, const int64_t* rows,
                      int64_t n_rows, double* out, double* delta_out, int nthreads) {
  const dao_problem P = *Pp;
  const int64_t* cu = P.cu;
  const int B = P.B, Hq = P.Hq, d = P.d;
  const int64_t Lmax = max_len(&P);
  int err = DAO_OK;
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#else
  (void)nthreads;
#endif
#pragma omp parallel
  {
    double* x = (double*)malloc(sizeof(double) * (size_t)(Lmax + 1) + (size_t)(Lmax / DAO_TILE + 1));
    double* sp_i = (double*)malloc(sizeof(double) * (size_t)d);
    double* sp_a = (double*)malloc(sizeof(double) * (size_t)d);
    double* dn_a = (double*)malloc(sizeof(double) * (size_t)d);
    /* the anchor rows sp_a, dn_a last evaluated by this thread: rows listed
     * group after group reuse them (the same values, evaluated once) */
    int cb = -1, ch = -1;
    int64_t ca = -1;
#pragma omp for schedule(dynamic, 64)
    for (int64_t it = 0; it < n_rows; ++it) {
      if (!x || !sp_i || !sp_a || !dn_a) {
#pragma omp atomic write
        err = DAO_ERR_NOMEM;
        continue;
      }
      const int b = (int)rows[3 * it];
      const int h = (int)rows[3 * it + 1];
      const int64_t i = rows[3 * it + 2];
      if (b < 0 || b >= B || h < 0 || h >= Hq || i < 0 || i >= cu[b + 1] - cu[b]) {
#pragma omp atomic write
        err = DAO_ERR_ARG;
        continue;
      }
      const int64_t L = cu[b + 1] - cu[b];
      const int64_t Lc = (L / gamma) * gamma;
      double* o = out + it * d;
      if (i >= Lc) { /* tail row: dense */
        attn_row(&P, DAO_MODE_DENSE, b, h, i, o, NULL, NULL, NULL, x);
        if (delta_out)
          for (int c = 0; c < d; ++c) delta_out[it * d + c] = 0.0;
        continue;
      }
      const int64_t a = (i / gamma) * gamma;
      attn_row(&P, smode, b, h, i, sp_i, NULL, NULL, NULL, x);   /* (A*V)_i */
      if (b != cb || h != ch || a != ca) {
        attn_row(&P, smode, b, h, a, sp_a, NULL, NULL, NULL, x);   /* (A*V)_a */
        attn_row(&P, DAO_MODE_DENSE, b, h, a, dn_a, NULL, NULL, NULL, x);    /* (A~V)_a */
        cb = b;
        ch = h;
        ca = a;
      }
      for (int c = 0; c < d; ++c) {
        const double dl = dn_a[c] - sp_a[c];
        o[c] = sp_i[c] + dl;
        if (delta_out) delta_out[it * d + c] = dl;
      }
    }
    free(x);
    free(sp_i);
    free(sp_a);
    free(dn_a);
  }
  return err;
}

int dao_delta_attention_rows(const void* q, const void* k, const void* v, int in_bf16,
                             const int64_t* cu, int B, int Hq, int Hkv, int d,
                             int window, int n_sink, int gamma,
                             const int64_t* rows, int64_t n_rows,
                             double* out, double* delta_out, int nthreads) {
  dao_problem P = {q, k, v, in_bf16, cu, B, Hq, Hkv, d, window, n_sink, NULL, NULL, 0, 0};
  if (check_problem(&P) != DAO_OK || !out || !rows || gamma < 1) return DAO_ERR_ARG;
  return delta_rows(&P, DAO_MODE_SPARSE, gamma, rows, n_rows, out, delta_out, nthreads);
}

/*
 * Correction variants (Sec. 3 "recompute", Eq. 5; interpolation appendix and
 * its algorithm for the alpha-beta-gamma filter).  Steps 1-4 of Algorithm 1
 * are as in dao_delta_attention: A*V for every row, A~V at the anchors,
 * Delta_i = A~V_{a_i} - (A*V)_{a_i} for anchor a_i = i*gamma.  Step 5 adds a
 * per-row correction c_r to (A*V)_r for r < L_c instead of repeat(Delta):
 *   DAO_CORR_DELTA      c_r = Delta_{floor(r/gamma)}                  (Eq. 6)
 *   DAO_CORR_RECOMPUTE  c_r = Delta_i if r = a_i, else 0               (Eq. 5)
 *   DAO_CORR_INTERP     c_{a_i+k} = (1 - beta_k) Delta_i + beta_k Delta_{i+1},
 *                       beta_k = k/(gamma-1) rising from 0 to 1 over the
 *                       group (0 when gamma = 1); the last group has no
 *                       successor and keeps Delta_i
 *   DAO_CORR_EMA        D = repeat(Delta, gamma); E_r = (1-b) E_{r-1} + b D_r
 *                       with E_{-1} = D_0, b = p0; c_r = E_r
 *   DAO_CORR_ABG        alpha-beta-gamma filter over the sequence Delta_0..,
 *                       in state-space form (see below): o_i is the filtered
 *                       position after Delta_i; c_r = o_{floor(r/gamma)}
 * Rows past L_c take the dense result as in the other entry points.  Every
 * operation is elementwise over the d channels.
 */
#define DAO_CORR_DELTA 0
#define DAO_CORR_RECOMPUTE 1
#define DAO_CORR_INTERP 2
#define DAO_CORR_EMA 3
#define DAO_CORR_ABG 4

int dao_delta_attention_variant(const void* q, const void* k, const void* v, int in_bf16,
                                const int64_t* cu, int B, int Hq, int Hkv, int d,
                                int window, int n_sink, int gamma, int mode,
                                double p0, double p1, double p2,
                                double* out, int nthreads) {
  dao_problem P = {q, k, v, in_bf16, cu, B, Hq, Hkv, d, window, n_sink, NULL, NULL, 0, 0};
  if (check_problem(&P) != DAO_OK || !out || gamma < 1) return DAO_ERR_ARG;
  if (mode < DAO_CORR_DELTA || mode > DAO_CORR_ABG) return DAO_ERR_ARG;
  const int64_t Lmax = max_len(&P);
  int err = DAO_OK;
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#else
  (void)nthreads;
#endif
#pragma omp parallel
  {
    double* x = (double*)malloc(sizeof(double) * (size_t)(Lmax + 1) + (size_t)(Lmax / DAO_TILE + 1));
    double* sp = (double*)malloc(sizeof(double) * (size_t)((Lmax + 1) * d));
    double* dl = (double*)malloc(sizeof(double) * (size_t)((Lmax / gamma + 1) * d));
    double* cr = (double*)malloc(sizeof(double) * (size_t)d);
    double* st = (double*)malloc(sizeof(double) * (size_t)(3 * d));
#pragma omp for schedule(dynamic, 1) collapse(2)
    for (int b = 0; b < B; ++b) {
      for (int h = 0; h < Hq; ++h) {
        if (!x || !sp || !dl || !cr || !st) {
#pragma omp atomic write
          err = DAO_ERR_NOMEM;
          continue;
        }
        const int64_t L = cu[b + 1] - cu[b];
        const int64_t nA = L / gamma;
        const int64_t Lc = nA * gamma;
        /* Step 1: A*V for every row of this sequence and head. */
        for (int64_t i = 0; i < L; ++i)
          attn_row(&P, DAO_MODE_SPARSE, b, h, i, sp + i * d, NULL, NULL, NULL, x);
        /* Steps 2-4: Delta_i at every anchor a_i = i*gamma < Lc. */
        for (int64_t i = 0; i < nA; ++i) {
          attn_row(&P, DAO_MODE_DENSE, b, h, i * gamma, cr, NULL, NULL, NULL, x);
          for (int c = 0; c < d; ++c) dl[i * d + c] = cr[c] - sp[i * gamma * d + c];
        }
        /* The interpolation appendix's alpha-beta-gamma filter, as a
         * state-space recursion over the anchors (unit step): state
         * s = (position, velocity, acceleration), constant-acceleration
         * transition F, the position observed, gain g = (p0, p1, p2):
         *   predict s^ = F s,  residual e = Delta_i - s^_0,  update s = s^ + g e,
         * from s = (Delta_0, 0, 0); Delta_i is replaced by the position. */
        if (mode == DAO_CORR_ABG && nA > 0) {
          static const double F[3][3] = {{1.0, 1.0, 0.5}, {0.0, 1.0, 1.0}, {0.0, 0.0, 1.0}};
          const double g[3] = {p0, p1, p2};
          double* sv = st; /* [3][d]: component r of channel c at sv[r * d + c] */
          for (int c = 0; c < d; ++c) { sv[c] = dl[c]; sv[d + c] = 0.0; sv[2 * d + c] = 0.0; }
          for (int64_t i = 1; i < nA; ++i) {
            for (int c = 0; c < d; ++c) {
              double sh[3];
              for (int r = 0; r < 3; ++r)
                sh[r] = F[r][0] * sv[c] + F[r][1] * sv[d + c] + F[r][2] * sv[2 * d + c];
              const double e = dl[i * d + c] - sh[0];
              for (int r = 0; r < 3; ++r) sv[r * d + c] = sh[r] + g[r] * e;
              dl[i * d + c] = sv[c];
            }
          }
        }
        /* Step 5 with the chosen correction, rows r < Lc */
        double* ema = st; /* E_{r-1} */
        if (mode == DAO_CORR_EMA && nA > 0)
          for (int c = 0; c < d; ++c) ema[c] = dl[c];
        for (int64_t r = 0; r < Lc; ++r) {
          const int64_t i = r / gamma, kk = r % gamma;
          for (int c = 0; c < d; ++c) {
            double corr;
            switch (mode) {
              case DAO_CORR_RECOMPUTE:
                corr = (kk == 0) ? dl[i * d + c] : 0.0;
                break;
              case DAO_CORR_INTERP: {
                const double beta = (gamma > 1) ? (double)kk / (double)(gamma - 1) : 0.0;
                const double next = (i + 1 < nA) ? dl[(i + 1) * d + c] : dl[i * d + c];
                corr = (1.0 - beta) * dl[i * d + c] + beta * next;
                break;
              }
              case DAO_CORR_EMA:
                ema[c] = (1.0 - p0) * ema[c] + p0 * dl[i * d + c];
                corr = ema[c];
                break;
              default: /* DELTA and the filtered ABG sequence */
                corr = dl[i * d + c];
            }
            out[((cu[b] + r) * Hq + h) * (int64_t)d + c] = sp[r * d + c] + corr;
          }
        }
        /* Tail rows: dense (implementation-details appendix). */
        for (int64_t r = Lc; r < L; ++r)
          attn_row(&P, DAO_MODE_DENSE, b, h, r, out + ((cu[b] + r) * Hq + h) * (int64_t)d,
                   NULL, NULL, NULL, x);
      }
    }
    free(x);
    free(sp);
    free(dl);
    free(cr);
    free(st);
  }
  return err;
}

/*
 * f* given by key-block lists (see the header comment): the lists are CSR,
 * ptr [B][Hkv][nqb + 1] (offsets into idx, non-decreasing per (b, g)) and
 * idx (key tile indices local to the sequence); nqb >= ceil(L / block_q)
 * for every sequence; block_q a positive multiple of 64.
 */
static int check_blocks(const dao_problem* P) {
  if (!P->blk_ptr || P->nqb < 1 || P->block_q < DAO_TILE || P->block_q % DAO_TILE != 0)
    return DAO_ERR_ARG;
  for (int b = 0; b < P->B; ++b) {
    const int64_t L = P->cu[b + 1] - P->cu[b];
    if ((L + P->block_q - 1) / P->block_q > P->nqb) return DAO_ERR_ARG;
    for (int g = 0; g < P->Hkv; ++g) {
      const int64_t* ptr = P->blk_ptr + ((int64_t)b * P->Hkv + g) * (P->nqb + 1);
      for (int qb = 0; qb < P->nqb; ++qb)
        if (ptr[qb + 1] < ptr[qb] || ptr[qb] < 0) return DAO_ERR_ARG;
      if (ptr[P->nqb] > ptr[0] && !P->blk_idx) return DAO_ERR_ARG;
    }
  }
  return DAO_OK;
}

/* Sparse attention under the block lists for every row (rows == NULL; out
 * [T, Hq, d]) or for n_rows triples (b, h, i) (out [n_rows, d]). */
int dao_block_attention(const void* q, const void* k, const void* v, int in_bf16,
                        const int64_t* cu, int B, int Hq, int Hkv, int d,
                        const int64_t* blk_ptr, const int64_t* blk_idx, int nqb, int block_q,
                        const int64_t* rows, int64_t n_rows, double* out, int nthreads) {
  dao_problem P = {q, k, v, in_bf16, cu, B, Hq, Hkv, d, 1, 0, blk_ptr, blk_idx, nqb, block_q};
  if (check_problem(&P) != DAO_OK || check_blocks(&P) != DAO_OK || !out) return DAO_ERR_ARG;
  const int64_t T = cu[B];
  const int64_t Lmax = max_len(&P);
  const int64_t n_items = rows ? n_rows : T * Hq;
  int err = DAO_OK;
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#else
  (void)nthreads;
#endif
#pragma omp parallel
  {
    double* x = (double*)malloc(sizeof(double) * (size_t)(Lmax + 1) + (size_t)(Lmax / DAO_TILE + 1));
#pragma omp for schedule(dynamic, 16)
    for (int64_t it = 0; it < n_items; ++it) {
      if (!x) {
#pragma omp atomic write
        err = DAO_ERR_NOMEM;
        continue;
      }
      int b = 0, h;
      int64_t i;
      if (rows) {
        b = (int)rows[3 * it];
        h = (int)rows[3 * it + 1];
        i = rows[3 * it + 2];
      } else {
        const int64_t t = it / Hq;
        h = (int)(it % Hq);
        while (cu[b + 1] <= t) ++b;
        i = t - cu[b];
      }
      if (b < 0 || b >= B || h < 0 || h >= Hq || i < 0 || i >= cu[b + 1] - cu[b]) {
#pragma omp atomic write
        err = DAO_ERR_ARG;
        continue;
      }
      attn_row(&P, DAO_MODE_BLOCKS, b, h, i, out + it * d, NULL, NULL, NULL, x);
    }
    free(x);
  }
  return err;
}

/* Algorithm 1 with f* from the block lists: out [T, Hq, d]; sparse and
 * delta optional as in dao_delta_attention. */
int dao_block_delta_attention(const void* q, const void* k, const void* v, int in_bf16,
                              const int64_t* cu, int B, int Hq, int Hkv, int d,
                              const int64_t* blk_ptr, const int64_t* blk_idx, int nqb,
                              int block_q, int gamma, double* out, double* sparse_out,
                              double* delta_out, int nthreads) {
  dao_problem P = {q, k, v, in_bf16, cu, B, Hq, Hkv, d, 1, 0, blk_ptr, blk_idx, nqb, block_q};
  if (check_problem(&P) != DAO_OK || check_blocks(&P) != DAO_OK || !out || gamma < 1)
    return DAO_ERR_ARG;
  return delta_full(&P, DAO_MODE_BLOCKS, gamma, out, sparse_out, delta_out, nthreads);
}

/* Algorithm 1 with f* from the block lists at selected rows (b, h, i). */
int dao_block_delta_attention_rows(const void* q, const void* k, const void* v, int in_bf16,
                                   const int64_t* cu, int B, int Hq, int Hkv, int d,
                                   const int64_t* blk_ptr, const int64_t* blk_idx, int nqb,
                                   int block_q, int gamma, const int64_t* rows, int64_t n_rows,
                                   double* out, double* delta_out, int nthreads) {
  dao_problem P = {q, k, v, in_bf16, cu, B, Hq, Hkv, d, 1, 0, blk_ptr, blk_idx, nqb, block_q};
  if (check_problem(&P) != DAO_OK || check_blocks(&P) != DAO_OK || !out || !rows || gamma < 1)
    return DAO_ERR_ARG;
  return delta_rows(&P, DAO_MODE_BLOCKS, gamma, rows, n_rows, out, delta_out, nthreads);
}

/* Softmax weights of one row (b, h, i) under the block lists (w[j], j <= i). */
int dao_block_attention_weights(const void* q, const void* k, const void* v, int in_bf16,
                                const int64_t* cu, int B, int Hq, int Hkv, int d,
                                const int64_t* blk_ptr, const int64_t* blk_idx, int nqb,
                                int block_q, int b, int h, int64_t i, double* w, double* o) {
  dao_problem P = {q, k, v, in_bf16, cu, B, Hq, Hkv, d, 1, 0, blk_ptr, blk_idx, nqb, block_q};
  if (check_problem(&P) != DAO_OK || check_blocks(&P) != DAO_OK || !w || !o) return DAO_ERR_ARG;
  if (b < 0 || b >= B || h < 0 || h >= Hq || i < 0 || i >= cu[b + 1] - cu[b]) return DAO_ERR_ARG;
  double* x = (double*)malloc(sizeof(double) * (size_t)(i + 1) + (size_t)(i / DAO_TILE + 1));
  if (!x) return DAO_ERR_NOMEM;
  attn_row(&P, DAO_MODE_BLOCKS, b, h, i, o, NULL, NULL, w, x);
  free(x);
  return DAO_OK;
}

/* Number of OpenMP threads a parallel region would use (1 without OpenMP). */
int dao_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

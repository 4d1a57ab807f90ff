/*
 * Runs the oracle's entry points on small seeded problems (fp64 and bfloat16
 * inputs, varlen, GQA, a dense tail, every correction variant, key-block lists
 * with entries the key set skips) and a few invalid calls.  Built with
 * AddressSanitizer and UndefinedBehaviorSanitizer by tests/test_sanitizers.py;
 * exits 0 when every call returns what it should.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int dao_attention(const void*, const void*, const void*, int, const int64_t*, int, int, int, int,
                  int, int, int, const int64_t*, int64_t, double*, double*, double*, int);
int dao_delta_attention(const void*, const void*, const void*, int, const int64_t*, int, int,
                        int, int, int, int, int, double*, double*, double*, int);
int dao_delta_attention_rows(const void*, const void*, const void*, int, const int64_t*, int,
                             int, int, int, int, int, int, const int64_t*, int64_t, double*,
                             double*, int);
int dao_delta_attention_variant(const void*, const void*, const void*, int, const int64_t*, int,
                                int, int, int, int, int, int, int, double, double, double,
                                double*, int);
int dao_block_delta_attention(const void*, const void*, const void*, int, const int64_t*, int,
                              int, int, int, const int64_t*, const int64_t*, int, int, int,
                              double*, double*, double*, int);
int dao_block_delta_attention_rows(const void*, const void*, const void*, int, const int64_t*,
                                   int, int, int, int, const int64_t*, const int64_t*, int, int,
                                   int, const int64_t*, int64_t, double*, double*, int);

static uint64_t rng = 88172645463325252ull;
static double uniform(void) { rng ^= rng << 13; rng ^= rng >> 7; rng ^= rng << 17; return (double)(rng >> 11) / 9007199254740992.0; }
static double gauss(void) { return sqrt(-2.0 * log(uniform() + 1e-300)) * cos(6.283185307179586 * uniform()); }

static int failures = 0;
static void expect(int got, int want, const char* what) {
  if (got != want) { fprintf(stderr, "%s: returned %d, expected %d\n", what, got, want); ++failures; }
}
static void finite(const double* x, int64_t n, const char* what) {
  for (int64_t i = 0; i < n; ++i)
    if (!isfinite(x[i])) { fprintf(stderr, "%s: non-finite value at %lld\n", what, (long long)i); ++failures; return; }
}

int main(void) {
  const int B = 3, Hq = 4, Hkv = 2, d = 16, window = 20, n_sink = 3;
  const int64_t cu[4] = {0, 150, 151, 300};  /* lengths 150, 1, 149 */
  const int64_t T = cu[B];
  double* q = malloc(sizeof(double) * T * Hq * d);
  double* k = malloc(sizeof(double) * T * Hkv * d);
  double* v = malloc(sizeof(double) * T * Hkv * d);
  uint16_t *qb = malloc(2 * T * Hq * d), *kb = malloc(2 * T * Hkv * d), *vb = malloc(2 * T * Hkv * d);
  for (int64_t i = 0; i < T * Hq * d; ++i) { q[i] = gauss(); float f = (float)q[i]; uint32_t u; memcpy(&u, &f, 4); qb[i] = (uint16_t)(u >> 16); }
  for (int64_t i = 0; i < T * Hkv * d; ++i) {
    k[i] = gauss(); v[i] = gauss();
    float f = (float)k[i]; uint32_t u; memcpy(&u, &f, 4); kb[i] = (uint16_t)(u >> 16);
    f = (float)v[i]; memcpy(&u, &f, 4); vb[i] = (uint16_t)(u >> 16);
  }
  double* out = malloc(sizeof(double) * T * Hq * d);
  double* sp = malloc(sizeof(double) * T * Hq * d);
  double* dl = malloc(sizeof(double) * T * Hq * d);
  double* m = malloc(sizeof(double) * T * Hq);
  double* z = malloc(sizeof(double) * T * Hq);
  int64_t rows[3 * 6] = {0, 0, 0, 0, 3, 149, 1, 1, 0, 2, 2, 64, 2, 0, 148, 0, 1, 47};
  double* ro = malloc(sizeof(double) * 6 * d);

  for (int bf = 0; bf < 2; ++bf) {
    const void *Q = bf ? (const void*)qb : q, *K = bf ? (const void*)kb : k, *V = bf ? (const void*)vb : v;
    for (int mode = 0; mode < 2; ++mode) {
      expect(dao_attention(Q, K, V, bf, cu, B, Hq, Hkv, d, window, n_sink, mode, NULL, 0, out, m, z, 2), 0, "attention");
      finite(out, T * Hq * d, "attention");
      expect(dao_attention(Q, K, V, bf, cu, B, Hq, Hkv, d, window, n_sink, mode, rows, 6, ro, NULL, NULL, 2), 0, "attention rows");
    }
    for (int gamma = 1; gamma <= 40; gamma += 13) {
      expect(dao_delta_attention(Q, K, V, bf, cu, B, Hq, Hkv, d, window, n_sink, gamma, out, sp, dl, 2), 0, "delta");
      finite(out, T * Hq * d, "delta");
      expect(dao_delta_attention_rows(Q, K, V, bf, cu, B, Hq, Hkv, d, window, n_sink, gamma, rows, 6, ro, NULL, 2), 0, "delta rows");
      for (int mode = 0; mode <= 4; ++mode) {
        expect(dao_delta_attention_variant(Q, K, V, bf, cu, B, Hq, Hkv, d, window, n_sink, gamma, mode, 0.3, 0.05, 0.01, out, 2), 0, "variant");
        finite(out, T * Hq * d, "variant");
      }
    }
    /* key-block lists, query blocks of 128 rows (nqb = 2), with skipped entries */
    const int nqb = 2, block_q = 128;
    int64_t ptr[3 * 2 * 3];
    int64_t idx[64];
    int n = 0;
    for (int b = 0; b < B; ++b)
      for (int g = 0; g < Hkv; ++g) {
        for (int qb_ = 0; qb_ < nqb; ++qb_) {
          ptr[(b * Hkv + g) * (nqb + 1) + qb_] = n;
          if (qb_ == 1) { idx[n++] = -3; idx[n++] = 0; idx[n++] = 1; idx[n++] = 2; idx[n++] = 9; }
        }
        ptr[(b * Hkv + g) * (nqb + 1) + nqb] = n;
      }
    expect(dao_block_delta_attention(Q, K, V, bf, cu, B, Hq, Hkv, d, ptr, idx, nqb, block_q, 16, out, sp, dl, 2), 0, "block delta");
    finite(out, T * Hq * d, "block delta");
    expect(dao_block_delta_attention_rows(Q, K, V, bf, cu, B, Hq, Hkv, d, ptr, idx, nqb, block_q, 16, rows, 6, ro, NULL, 2), 0, "block rows");
    /* invalid calls */
    expect(dao_block_delta_attention(Q, K, V, bf, cu, B, Hq, Hkv, d, ptr, idx, 1, block_q, 16, out, NULL, NULL, 2), 1, "block nqb too small");
    expect(dao_delta_attention(Q, K, V, bf, cu, B, Hq, 3, d, window, n_sink, 16, out, NULL, NULL, 2), 1, "Hq % Hkv");
    expect(dao_delta_attention(Q, K, V, bf, cu, B, Hq, Hkv, d, 0, n_sink, 16, out, NULL, NULL, 2), 1, "window 0");
  }
  free(q); free(k); free(v); free(qb); free(kb); free(vb);
  free(out); free(sp); free(dl); free(m); free(z); free(ro);
  if (failures) { fprintf(stderr, "%d failures\n", failures); return 1; }
  printf("oracle driver ok\n");
  return 0;
}

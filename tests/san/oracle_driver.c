/* The fp64 oracle under AddressSanitizer and UndefinedBehaviorSanitizer:
 * forward and backward of both nodes on tiny seeded problems (n = 1, 2, 5,
 * 9), with no mask, a random mask and a fully masked map, over every row
 * and over row and bias-query subsets; and the fused layer-norm + linear
 * oracle.  Exits non-zero if an output that must be finite is not. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

void oracle_fwd(int node, int64_t n, int64_t H, int64_t d, double scale, const double* q,
                const double* k, const double* v, const double* gate, const double* bias,
                const uint8_t* mask, double* out, double* lse, const int64_t* rows,
                int64_t nrows);
void oracle_bwd(int node, int64_t n, int64_t H, int64_t d, double scale, const double* q,
                const double* k, const double* v, const double* gate, const double* bias,
                const uint8_t* mask, const double* dout, double* dq, double* dk, double* dv,
                double* dg, double* db, const int64_t* rows, int64_t nrows,
                const int64_t* dbq, int64_t ndbq);

void oracle_lnl_fwd(int64_t M, int64_t K, int64_t N, double eps, const double* x,
                    const double* gamma, const double* beta, const double* w, double* o2,
                    double* mean, double* rstd, const int64_t* rows, int64_t nrows);
void oracle_lnl_bwd(int64_t M, int64_t K, int64_t N, double eps, const double* x,
                    const double* gamma, const double* beta, const double* w, const double* do2,
                    double* dx, double* dw, double* dgamma, double* dbeta, const int64_t* rows,
                    int64_t nrows);

static uint64_t state = 0x9e3779b97f4a7c15ull;
static double uni(void) {  /* splitmix64 -> [-1, 1) */
  uint64_t z = (state += 0x9e3779b97f4a7c15ull);
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  z ^= z >> 31;
  return (double)(z >> 11) / 4503599627370496.0 - 1.0;
}

static double* arr(int64_t count) {
  double* p = (double*)malloc(sizeof(double) * (size_t)count);
  for (int64_t i = 0; i < count; ++i) p[i] = uni();
  return p;
}

int main(void) {
  int bad = 0;
  const int64_t ns[] = {1, 2, 5, 9};
  for (int in = 0; in < 4; ++in) {
    const int64_t n = ns[in], H = 2, d = 4, pair = n * n * H * d, bias = n * n * H;
    double *q = arr(pair), *k = arr(pair), *v = arr(pair), *g = arr(pair), *b = arr(bias),
           *dout = arr(pair);
    double *out = arr(pair), *lse = arr(bias), *dq = arr(pair), *dk = arr(pair),
           *dv = arr(pair), *dg = arr(pair), *db = arr(bias);
    uint8_t* mask = (uint8_t*)malloc((size_t)(n * n));
    for (int mk = 0; mk < 3; ++mk) {
      for (int64_t i = 0; i < n * n; ++i) mask[i] = mk == 2 ? 0 : (uni() > -0.6);
      const uint8_t* mp = mk == 0 ? NULL : mask;
      for (int node = 0; node < 2; ++node) {
        oracle_fwd(node, n, H, d, 0.5, q, k, v, g, b, mp, out, lse, NULL, 0);
        oracle_bwd(node, n, H, d, 0.5, q, k, v, g, b, mp, dout, dq, dk, dv, dg, db, NULL, 0,
                   NULL, 0);
        for (int64_t i = 0; i < pair; ++i)
          if (!isfinite(out[i]) || !isfinite(dq[i]) || !isfinite(dk[i]) || !isfinite(dv[i]) ||
              !isfinite(dg[i]))
            ++bad;
        for (int64_t i = 0; i < bias; ++i)
          if (!isfinite(db[i])) ++bad;
        const int64_t rows[2] = {n - 1, 0}, qs[1] = {n / 2};
        oracle_fwd(node, n, H, d, 0.5, q, k, v, g, b, mp, out, lse, rows, n > 1 ? 2 : 1);
        oracle_bwd(node, n, H, d, 0.5, q, k, v, g, b, mp, dout, dq, dk, dv, dg, db, rows,
                   n > 1 ? 2 : 1, qs, 1);
      }
    }
    free(q); free(k); free(v); free(g); free(b); free(dout); free(out); free(lse);
    free(dq); free(dk); free(dv); free(dg); free(db); free(mask);
  }
  {
    const int64_t M = 7, K = 16, N = 12;
    double *x = arr(M * K), *gm = arr(K), *bt = arr(K), *w = arr(K * N), *do2 = arr(M * N);
    double *o2 = arr(M * N), *mean = arr(M), *rstd = arr(M), *dx = arr(M * K), *dw = arr(K * N),
           *dgm = arr(K), *dbt = arr(K);
    const int64_t rows[3] = {6, 0, 3};
    oracle_lnl_fwd(M, K, N, 1e-5, x, gm, bt, w, o2, mean, rstd, NULL, 0);
    oracle_lnl_fwd(M, K, N, 1e-5, x, gm, bt, w, o2, mean, rstd, rows, 3);
    oracle_lnl_bwd(M, K, N, 1e-5, x, gm, bt, w, do2, dx, dw, dgm, dbt, NULL, 0);
    oracle_lnl_bwd(M, K, N, 1e-5, x, gm, bt, w, do2, dx, NULL, NULL, NULL, rows, 3);
    for (int64_t i = 0; i < M * N; ++i) bad += !isfinite(o2[i]);
    for (int64_t i = 0; i < K * N; ++i) bad += !isfinite(dw[i]);
    for (int64_t i = 0; i < M * K; ++i) bad += !isfinite(dx[i]);
    free(x); free(gm); free(bt); free(w); free(do2); free(o2); free(mean); free(rstd);
    free(dx); free(dw); free(dgm); free(dbt);
  }
  printf("oracle driver: %d non-finite outputs\n", bad);
  return bad == 0 ? 0 : 1;
}

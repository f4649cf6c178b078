/*
 * Fused layer-norm + linear projection oracle: plain fp64 CPU reference.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may call, link or
 * load this file; only the tests and the benchmark's CPU-baseline leg use
 * it.  It shares no code, header, table or constant with the GPU library.
 *
 * What it computes (MegaFold, arXiv 2506.20686, Section IV "fused
 * layer-norm & linear projection" and the appendix table of fused
 * AlphaFold operators), for every row m of x [M][K]:
 *   mean = sum_k x / K,  var = sum_k (x - mean)^2 / K   (biased variance)
 *   rstd = 1 / sqrt(var + eps),  xhat = (x - mean) rstd
 *   o1 = xhat * gamma + beta,    o2 = o1 W            (W [K][N], no bias)
 * Backward, given do2 = dL/do2 [M][N] (appendix table):
 *   do1 = do2 W^T,  dW = o1^T do2,  dgamma = sum_m do1 * xhat,
 *   dbeta = sum_m do1,  wdy = do1 * gamma,
 *   c1 = sum_k xhat * wdy / K,  c2 = sum_k wdy / K,
 *   dx = rstd (wdy - c1 xhat - c2).
 * Readings where the paper's table is loose: the table writes 1/Var where
 * the listing (and the calculus) uses rstd; the mean in c1 and c2 runs over
 * the K features of a row (the listing divides by K); dgamma and dbeta are
 * summed over rows; the paper's atomic adds become plain fixed-order sums.
 *
 * Plain loops in the order of the formulas above; rows run in parallel
 * (OpenMP) where each row's results are independent, and the sums over rows
 * (dW, dgamma, dbeta) run in row order.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>

/* Row statistics and o1 for one row. */
static void ln_row(int64_t K, const double* x, const double* gamma, const double* beta,
                   double eps, double* mean_out, double* rstd_out, double* xhat, double* o1) {
  double mean = 0.0;
  for (int64_t k = 0; k < K; ++k) mean += x[k];
  mean /= (double)K;
  double var = 0.0;
  for (int64_t k = 0; k < K; ++k) var += (x[k] - mean) * (x[k] - mean);
  var /= (double)K;
  const double rstd = 1.0 / sqrt(var + eps);
  for (int64_t k = 0; k < K; ++k) {
    xhat[k] = (x[k] - mean) * rstd;
    o1[k] = xhat[k] * gamma[k] + beta[k];
  }
  *mean_out = mean;
  *rstd_out = rstd;
}

/* Forward.  rows / nrows: only those rows (NULL = all M); other rows are
 * left untouched.  o2 [M][N], mean and rstd [M]. */
void oracle_lnl_fwd(int64_t M, int64_t K, int64_t N, double eps, const double* x,
                    const double* gamma, const double* beta, const double* w, double* o2,
                    double* mean, double* rstd, const int64_t* rows, int64_t nrows) {
  const int64_t cnt = rows ? nrows : M;
#pragma omp parallel for schedule(dynamic, 16)
  for (int64_t i = 0; i < cnt; ++i) {
    const int64_t m = rows ? rows[i] : i;
    double* xhat = (double*)malloc(sizeof(double) * K);
    double* o1 = (double*)malloc(sizeof(double) * K);
    ln_row(K, x + m * K, gamma, beta, eps, &mean[m], &rstd[m], xhat, o1);
    for (int64_t n = 0; n < N; ++n) {
      double s = 0.0;
      for (int64_t k = 0; k < K; ++k) s += o1[k] * w[k * N + n];
      o2[m * N + n] = s;
    }
    free(xhat);
    free(o1);
  }
}

/* Backward.  dx [M][K] for the listed rows (NULL = all); dW [K][N], dgamma
 * and dbeta [K] over ALL rows (skipped when dw is NULL). */
void oracle_lnl_bwd(int64_t M, int64_t K, int64_t N, double eps, const double* x,
                    const double* gamma, const double* beta, const double* w, const double* do2,
                    double* dx, double* dw, double* dgamma, double* dbeta, const int64_t* rows,
                    int64_t nrows) {
  /* dx per row (independent rows) */
  const int64_t cnt = rows ? nrows : M;
#pragma omp parallel for schedule(dynamic, 16)
  for (int64_t i = 0; i < cnt; ++i) {
    const int64_t m = rows ? rows[i] : i;
    double* xhat = (double*)malloc(sizeof(double) * K);
    double* o1 = (double*)malloc(sizeof(double) * K);
    double* wdy = (double*)malloc(sizeof(double) * K);
    double mean, rstd;
    ln_row(K, x + m * K, gamma, beta, eps, &mean, &rstd, xhat, o1);
    double c1 = 0.0, c2 = 0.0;
    for (int64_t k = 0; k < K; ++k) {
      double d1 = 0.0; /* do1 = do2 W^T */
      for (int64_t n = 0; n < N; ++n) d1 += do2[m * N + n] * w[k * N + n];
      wdy[k] = d1 * gamma[k];
      c1 += xhat[k] * wdy[k];
      c2 += wdy[k];
    }
    c1 /= (double)K;
    c2 /= (double)K;
    for (int64_t k = 0; k < K; ++k) dx[m * K + k] = rstd * (wdy[k] - c1 * xhat[k] - c2);
    free(xhat);
    free(o1);
    free(wdy);
  }
  if (dw == NULL) return;
  /* dW, dgamma, dbeta: sums over all rows in row order.  Row statistics
   * first; then each k (one thread each) walks the rows in order. */
  double* mean = (double*)malloc(sizeof(double) * M);
  double* rstd = (double*)malloc(sizeof(double) * M);
#pragma omp parallel for schedule(static)
  for (int64_t m = 0; m < M; ++m) {
    double* xhat = (double*)malloc(sizeof(double) * K);
    double* o1 = (double*)malloc(sizeof(double) * K);
    ln_row(K, x + m * K, gamma, beta, eps, &mean[m], &rstd[m], xhat, o1);
    free(xhat);
    free(o1);
  }
#pragma omp parallel for schedule(static)
  for (int64_t k = 0; k < K; ++k) {
    for (int64_t n = 0; n < N; ++n) dw[k * N + n] = 0.0;
    double dg = 0.0, db = 0.0;
    for (int64_t m = 0; m < M; ++m) {
      const double xhat = (x[m * K + k] - mean[m]) * rstd[m];
      const double o1 = xhat * gamma[k] + beta[k];
      double d1 = 0.0; /* do1 = do2 W^T */
      for (int64_t n = 0; n < N; ++n) {
        dw[k * N + n] += o1 * do2[m * N + n];
        d1 += do2[m * N + n] * w[k * N + n];
      }
      dg += d1 * xhat;
      db += d1;
    }
    dgamma[k] = dg;
    dbeta[k] = db;
  }
  free(mean);
  free(rstd);
}

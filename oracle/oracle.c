/*
 * Triangle self-attention oracle: plain fp64 CPU reference.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may call, link or
 * load this file; only the tests, the smoke check and the CPU-baseline leg
 * of the benchmark use it.  It shares no code, header, table or constant
 * with the GPU library.
 *
 * What it computes (MegaFold, arXiv 2506.20686):
 *   - 3D attention over the pair representation, Section IV-A and the
 *     appendix table that lists EvoAttention's computations:
 *       S = Q K^T + Bias (bias broadcast over the pair-row axis),
 *       P = softmax(S) over the keys,  A = P V.
 *     The method (online softmax, Section IV-A) reaches this exact result,
 *     so the oracle is the plain two-pass definition, with no online
 *     rescaling, no tiling and no fusion.
 *   - A softmax scale multiplies Q K^T (the paper writes none; scale = 1
 *     reproduces it literally).
 *   - A sigmoid gate O = sigmoid(G) * A (AF3 triangle attention; the paper
 *     is silent on the gate).
 *   - The log-sum-exp saved for the backward pass (Section IV-A, last
 *     paragraph of the forward description): LSE = max + ln(sum exp).
 *   - Backward, appendix table, with the standard softmax algebra:
 *       dV = P^T dA,  dP = dA V^T,  D = rowsum(dA * A),
 *       dS = P * (dP - D),  dQ = scale dS K,  dK = scale dS^T Q,
 *       dBias = sum of dS over the broadcast (pair-row) axis.
 *     dA = dO * sigmoid(G) and dG = dO * A * sigmoid'(G) are the chain rule
 *     through the gate.
 *
 * Node variants (Section III-B and IV-B: the attention axis alternates
 * between stages).  Every pair tensor X is indexed X[a][b][h][c].
 *   starting node, output pair (r, q), key k:
 *       s_k = scale <Q[r][q], K[r][k]> + B[q][k],  valid iff mask[r][k],
 *       A   = sum_k P_k V[r][k],  O[r][q] = sigmoid(G[r][q]) * A.
 *   ending node, output pair (i, j), key k (the attention runs along the
 *   first pair axis, for a fixed second index j):
 *       s_k = scale <Q[i][j], K[k][j]> + B[k][i],  valid iff mask[k][j],
 *       A   = sum_k P_k V[k][j],  O[i][j] = sigmoid(G[i][j]) * A.
 *   The two are coded with their own index formulas below; the tests check
 *   that ending == T(starting(T x)) with T swapping the two pair axes.
 *
 * Masked keys are excluded exactly (weight 0).  A query with no valid key
 * gets A = 0, O = 0, LSE = -inf and contributes nothing to any gradient.
 *
 * Parity pins (see tests/test_oracle_pins.py): library SDPA and autograd in
 * float64, central finite differences, closed forms, invariants and
 * hand-derived fixtures.  The paper prints no numeric example.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define NODE_STARTING 0
#define NODE_ENDING 1

/* Offsets, in units of pair entries, of the operands that one
 * (node, row, query, key) triple touches.  Each node has its own formula. */
typedef struct {
  int node;
  int64_t n;
} geom;

/* pair (row, query) of the output; Q, G, O, dO, dQ, dG and LSE live here */
static int64_t at_query(geom g, int64_t row, int64_t qi) {
  if (g.node == NODE_STARTING) return row * g.n + qi; /* [r][q] */
  return qi * g.n + row;                              /* [i][j], j = row */
}
/* pair holding key k of a row; K, V, dK and dV live here */
static int64_t at_key(geom g, int64_t row, int64_t k) {
  if (g.node == NODE_STARTING) return row * g.n + k; /* [r][k] */
  return k * g.n + row;                              /* [k][j], j = row */
}
/* bias pair for (query, key) */
static int64_t at_bias(geom g, int64_t qi, int64_t k) {
  if (g.node == NODE_STARTING) return qi * g.n + k; /* B[q][k] */
  return k * g.n + qi;                              /* B[k][i] */
}
/* mask entry for (row, key) */
static int64_t at_mask(geom g, int64_t row, int64_t k) {
  if (g.node == NODE_STARTING) return row * g.n + k; /* mask[r][k] */
  return k * g.n + row;                              /* mask[k][j] */
}

static double sigmoid(double x) { return 1.0 / (1.0 + exp(-x)); }

typedef struct {
  geom g;
  int64_t H, d;
  double scale;
  const double *q, *k, *v, *gate, *bias;
  const uint8_t* mask;
} problem;

/* One query of one row and head: logits, probabilities and the ungated
 * output A.  s, p are length n; a is length d.  Returns the LSE (-inf when
 * no key is valid, in which case p and a are zero). */
static double attend(const problem* pb, int64_t row, int64_t qi, int64_t hh,
                     double* s, double* p, double* a) {
  const int64_t n = pb->g.n, H = pb->H, d = pb->d;
  const double* qv = pb->q + (at_query(pb->g, row, qi) * H + hh) * d;
  int any = 0;
  double mx = -INFINITY;
  for (int64_t k = 0; k < n; ++k) {
    int valid = pb->mask == NULL || pb->mask[at_mask(pb->g, row, k)] != 0;
    if (!valid) {
      s[k] = -INFINITY;
      continue;
    }
    const double* kv = pb->k + (at_key(pb->g, row, k) * H + hh) * d;
    double dot = 0.0;
    for (int64_t c = 0; c < d; ++c) dot += qv[c] * kv[c];
    s[k] = pb->scale * dot + pb->bias[at_bias(pb->g, qi, k) * H + hh];
    if (s[k] > mx) mx = s[k];
    any = 1;
  }
  for (int64_t c = 0; c < d; ++c) a[c] = 0.0;
  if (!any) {
    for (int64_t k = 0; k < n; ++k) p[k] = 0.0;
    return -INFINITY;
  }
  /* two-pass softmax: LSE = max + ln(sum exp(s - max)), P = exp(s - LSE) */
  double z = 0.0;
  for (int64_t k = 0; k < n; ++k)
    if (s[k] != -INFINITY) z += exp(s[k] - mx);
  const double lse = mx + log(z);
  for (int64_t k = 0; k < n; ++k) p[k] = (s[k] == -INFINITY) ? 0.0 : exp(s[k] - lse);
  for (int64_t k = 0; k < n; ++k) {
    if (p[k] == 0.0) continue;
    const double* vv = pb->v + (at_key(pb->g, row, k) * H + hh) * d;
    for (int64_t c = 0; c < d; ++c) a[c] += p[k] * vv[c];
  }
  return lse;
}

static int64_t* make_list(const int64_t* list, int64_t count, int64_t n, int64_t* out_count) {
  int64_t m = list ? count : n;
  int64_t* r = (int64_t*)malloc(sizeof(int64_t) * (size_t)(m > 0 ? m : 1));
  for (int64_t i = 0; i < m; ++i) r[i] = list ? list[i] : i;
  *out_count = m;
  return r;
}

/* Forward.  Pair tensors [n][n][h][d], bias [n][n][h], mask [n][n] (NULL =
 * all valid); out [n][n][h][d], lse [n][n][h].  rows/nrows restricts the work
 * to the listed rows (row = first pair axis for the starting node, second for
 * the ending node); NULL means every row.  Entries of other rows are left
 * untouched. */
void oracle_fwd(int node, int64_t n, int64_t H, int64_t d, double scale, const double* q,
                const double* k, const double* v, const double* gate, const double* bias,
                const uint8_t* mask, double* out, double* lse, const int64_t* rows,
                int64_t nrows) {
  problem pb = {{node, n}, H, d, scale, q, k, v, gate, bias, mask};
  int64_t m;
  int64_t* rl = make_list(rows, nrows, n, &m);
#pragma omp parallel
  {
    double* s = (double*)malloc(sizeof(double) * (size_t)n);
    double* p = (double*)malloc(sizeof(double) * (size_t)n);
    double* a = (double*)malloc(sizeof(double) * (size_t)d);
#pragma omp for schedule(dynamic)
    for (int64_t t = 0; t < m * H; ++t) {
      const int64_t row = rl[t / H], hh = t % H;
      for (int64_t qi = 0; qi < n; ++qi) {
        const int64_t at = at_query(pb.g, row, qi);
        lse[at * H + hh] = attend(&pb, row, qi, hh, s, p, a);
        for (int64_t c = 0; c < d; ++c) {
          const int64_t e = (at * H + hh) * d + c;
          out[e] = sigmoid(gate[e]) * a[c];
        }
      }
    }
    free(s);
    free(p);
    free(a);
  }
  free(rl);
}

/* Backward of L = sum(dout * out).  Gradients dq, dk, dv, dg [n][n][h][d] for
 * the listed rows (NULL = all; these entries are overwritten, others left
 * untouched) and the bias gradient db [n][n][h] for the listed query indices
 * (NULL = all): db is written at every bias entry (query in list, any key,
 * any head), i.e. db[q][k] for the starting node and db[k][i] for the
 * ending node.  The mask and the scale receive no gradient. */
void oracle_bwd(int node, int64_t n, int64_t H, int64_t d, double scale, const double* q,
                const double* k, const double* v, const double* gate, const double* bias,
                const uint8_t* mask, const double* dout, double* dq, double* dk, double* dv,
                double* dg, double* db, const int64_t* rows, int64_t nrows,
                const int64_t* dbq, int64_t ndbq) {
  problem pb = {{node, n}, H, d, scale, q, k, v, gate, bias, mask};
  int64_t m, mq;
  int64_t* rl = make_list(rows, nrows, n, &m);
  int64_t* ql = make_list(dbq, ndbq, n, &mq);

  /* Part 1: gradients that live on one row (dQ, dG on the row's queries,
   * dK, dV on the row's keys). */
#pragma omp parallel
  {
    double* s = (double*)malloc(sizeof(double) * (size_t)n);
    double* p = (double*)malloc(sizeof(double) * (size_t)n);
    double* a = (double*)malloc(sizeof(double) * (size_t)d);
    double* da = (double*)malloc(sizeof(double) * (size_t)d);
#pragma omp for schedule(dynamic)
    for (int64_t t = 0; t < m * H; ++t) {
      const int64_t row = rl[t / H], hh = t % H;
      for (int64_t kk = 0; kk < n; ++kk) {
        const int64_t e0 = (at_key(pb.g, row, kk) * H + hh) * d;
        for (int64_t c = 0; c < d; ++c) dk[e0 + c] = dv[e0 + c] = 0.0;
      }
      for (int64_t qi = 0; qi < n; ++qi) {
        attend(&pb, row, qi, hh, s, p, a);
        const int64_t e0 = (at_query(pb.g, row, qi) * H + hh) * d;
        /* through the gate: O = sigmoid(G) A */
        double dsum = 0.0;
        for (int64_t c = 0; c < d; ++c) {
          const double sg = sigmoid(gate[e0 + c]);
          da[c] = dout[e0 + c] * sg;
          dg[e0 + c] = dout[e0 + c] * a[c] * sg * (1.0 - sg);
          dsum += da[c] * a[c]; /* D = rowsum(dA * A) */
          dq[e0 + c] = 0.0;
        }
        for (int64_t kk = 0; kk < n; ++kk) {
          if (p[kk] == 0.0) continue;
          const int64_t ek = (at_key(pb.g, row, kk) * H + hh) * d;
          double dp = 0.0; /* dP = dA V^T */
          for (int64_t c = 0; c < d; ++c) dp += da[c] * v[ek + c];
          const double ds = p[kk] * (dp - dsum); /* dS = P (dP - D) */
          for (int64_t c = 0; c < d; ++c) {
            dq[e0 + c] += scale * ds * k[ek + c]; /* dQ = scale dS K */
            dk[ek + c] += scale * ds * q[e0 + c]; /* dK = scale dS^T Q */
            dv[ek + c] += p[kk] * da[c];          /* dV = P^T dA */
          }
        }
      }
    }
    free(s);
    free(p);
    free(a);
    free(da);
  }

  /* Part 2: dBias[q][k] = sum over rows of dS[row][q][k], rows in order. */
#pragma omp parallel
  {
    double* s = (double*)malloc(sizeof(double) * (size_t)n);
    double* p = (double*)malloc(sizeof(double) * (size_t)n);
    double* a = (double*)malloc(sizeof(double) * (size_t)d);
    double* da = (double*)malloc(sizeof(double) * (size_t)d);
    double* acc = (double*)malloc(sizeof(double) * (size_t)n);
#pragma omp for schedule(dynamic)
    for (int64_t t = 0; t < mq * H; ++t) {
      const int64_t qi = ql[t / H], hh = t % H;
      for (int64_t kk = 0; kk < n; ++kk) acc[kk] = 0.0;
      for (int64_t row = 0; row < n; ++row) {
        attend(&pb, row, qi, hh, s, p, a);
        const int64_t e0 = (at_query(pb.g, row, qi) * H + hh) * d;
        double dsum = 0.0;
        for (int64_t c = 0; c < d; ++c) {
          da[c] = dout[e0 + c] * sigmoid(gate[e0 + c]);
          dsum += da[c] * a[c];
        }
        for (int64_t kk = 0; kk < n; ++kk) {
          if (p[kk] == 0.0) continue;
          const int64_t ek = (at_key(pb.g, row, kk) * H + hh) * d;
          double dp = 0.0;
          for (int64_t c = 0; c < d; ++c) dp += da[c] * v[ek + c];
          acc[kk] += p[kk] * (dp - dsum);
        }
      }
      for (int64_t kk = 0; kk < n; ++kk) db[at_bias(pb.g, qi, kk) * H + hh] = acc[kk];
    }
    free(s);
    free(p);
    free(a);
    free(da);
    free(acc);
  }
  free(rl);
  free(ql);
}

/* Threads the oracle's parallel loops use (for reporting). */
int oracle_max_threads(void) { return omp_get_max_threads(); }

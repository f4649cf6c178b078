"""fp64 oracle of the fused transition layer (numpy).

TEST INFRASTRUCTURE ONLY: the product path never imports this module.

What is computed follows Section IV (fused layer-norm & linear projection,
fused SwiGLU, fused transition layer) and the appendix listing of the
transition layer's forward and backward passes.  For every row x of the pair
representation (C features):

  mean, rstd = mean and 1/sqrt(var + eps) of x (biased variance)
  o1   = (x - mean) * rstd * gamma + beta
  [a | b] = o1 W1                  W1 [C][2F]: a = first F columns, b = last F
  u    = a * sigmoid(a) * b        (SwiGLU)
  out  = u W2                      W2 [F][C]

and, for L = sum(dout * out), the backward pass:

  du   = dout W2^T
  dW2  = sum over rows of u^T dout
  da   = du * b * sigmoid(a) * (1 + a (1 - sigmoid(a)))
  db   = du * a * sigmoid(a)
  dh   = [da | db]
  dW1  = sum over rows of o1^T dh
  do1  = dh W1^T
  dgamma = sum over rows of do1 * xhat,  dbeta = sum over rows of do1
  wdy  = do1 * gamma,  c1 = mean over features of xhat * wdy,  c2 = mean of wdy
  dx   = rstd * (wdy - c1 * xhat - c2)

Rows are processed in blocks so that any number of rows fits in memory;
numpy's matmul is the only library step.
"""
import numpy as np

_BLOCK = 16384


def _f64(a):
    if hasattr(a, "detach"):
        a = a.detach().cpu().double().numpy()
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _sigmoid(a):
    return 1.0 / (1.0 + np.exp(-a))


def _ln(x, gamma, beta, eps):
    mean = x.mean(axis=1)
    var = ((x - mean[:, None]) ** 2).mean(axis=1)
    rstd = 1.0 / np.sqrt(var + eps)
    xhat = (x - mean[:, None]) * rstd[:, None]
    return xhat, xhat * gamma + beta, mean, rstd


def _blocks(m, rows):
    if rows is None:
        for r0 in range(0, m, _BLOCK):
            yield np.arange(r0, min(m, r0 + _BLOCK))
    else:
        rows = np.asarray(rows, dtype=np.int64)
        for r0 in range(0, rows.size, _BLOCK):
            yield rows[r0:r0 + _BLOCK]


def trn_fwd(x, gamma, beta, w1, w2, eps=1e-5, rows=None):
    """Forward: returns (out [M, C], mean [M], rstd [M]) in float64; rows
    restricts the work to those rows (other entries NaN)."""
    x, gamma, beta, w1, w2 = (_f64(t) for t in (x, gamma, beta, w1, w2))
    m, c = x.shape
    f = w2.shape[0]
    assert w1.shape == (c, 2 * f) and w2.shape == (f, c)
    out = np.full((m, c), np.nan)
    mean = np.full(m, np.nan)
    rstd = np.full(m, np.nan)
    for r in _blocks(m, rows):
        _, o1, mu, rs = _ln(x[r], gamma, beta, eps)
        h = o1 @ w1
        a, b = h[:, :f], h[:, f:]
        out[r] = (a * _sigmoid(a) * b) @ w2
        mean[r], rstd[r] = mu, rs
    return out, mean, rstd


def trn_bwd(x, gamma, beta, w1, w2, dout, eps=1e-5, rows=None, sums=True):
    """Backward of sum(dout * out): returns (dx [M, C], dw1 [C, 2F],
    dw2 [F, C], dgamma [C], dbeta [C]) in float64.  rows restricts dx to
    those rows (other entries NaN); the sums over rows always take every row
    (sums=False skips them: the four sums are then None)."""
    x, gamma, beta, w1, w2, dout = (_f64(t) for t in (x, gamma, beta, w1, w2, dout))
    m, c = x.shape
    f = w2.shape[0]
    dx = np.full((m, c), np.nan)
    dw1 = np.zeros((c, 2 * f)) if sums else None
    dw2 = np.zeros((f, c)) if sums else None
    dgamma = np.zeros(c) if sums else None
    dbeta = np.zeros(c) if sums else None
    want = None if rows is None else np.zeros(m, dtype=bool)
    if want is not None:
        want[np.asarray(rows, dtype=np.int64)] = True
    # every row when the sums are wanted, else only the requested rows
    for r in _blocks(m, None if (sums or rows is None) else rows):
        xhat, o1, _, rs = _ln(x[r], gamma, beta, eps)
        h = o1 @ w1
        a, b = h[:, :f], h[:, f:]
        sg = _sigmoid(a)
        silu = a * sg
        do = dout[r]
        du = do @ w2.T
        dh = np.concatenate([du * b * sg * (1.0 + a * (1.0 - sg)), du * silu], axis=1)
        do1 = dh @ w1.T
        if sums:
            dw2 += (silu * b).T @ do
            dw1 += o1.T @ dh
            dgamma += (do1 * xhat).sum(axis=0)
            dbeta += do1.sum(axis=0)
        wdy = do1 * gamma
        c1 = (xhat * wdy).mean(axis=1, keepdims=True)
        c2 = wdy.mean(axis=1, keepdims=True)
        d = rs[:, None] * (wdy - c1 * xhat - c2)
        if want is None:
            dx[r] = d
        else:
            sel = want[r]
            dx[r[sel]] = d[sel]
    return dx, dw1, dw2, dgamma, dbeta


def trn_sum_scales(x, gamma, beta, w1, w2, dout, eps=1e-5):
    """Error scales of the four sums over rows of trn_bwd (dW1, dW2, dgamma,
    dbeta) for an implementation that rounds its matrix operands to bf16 and
    forms the sums regrouped: dW1 = gamma G + beta s^T, dgamma = sum_c W1 o
    G, dbeta = W1 s with G = xhat^T dh and s = column sums of dh (o1 = xhat
    gamma + beta substituted), and dW2 = u^T dout.  Returns two tuples (S, R)
    of four arrays each.

    S: rounding errors of the terms of G, s and dW2 add up like the l2 norms
    over rows of those terms, carried into the regrouped results by |gamma|,
    |beta| and |W1|:
      dW1[k][c] : |gamma_k| sqrt(sum_r xhat^2 dh^2) + |beta_k| sqrt(sum_r dh^2)
      dW2[f][k] : sqrt(sum_r u^2 dout^2)
      dgamma[k] : sqrt(sum_c W1[k][c]^2 sum_r xhat^2 dh^2)
      dbeta[k]  : sqrt(sum_c W1[k][c]^2 sum_r dh^2)
    R: the same norms with dh and u replaced by the first-order change that
    the rounding of o1 to bf16 (relative 2^-9 per feature, independent) makes
    in them through a and b: da_err = 2^-9 sqrt(sum_k (o1_k W1[k][a col])^2),
    likewise for b, propagated by the derivatives of da, db and u in a and b.
    This term dominates where a factor of a term nearly vanishes (b close to
    0), which a sum over few rows does not average out."""
    x, gamma, beta, w1, w2, dout = (_f64(t) for t in (x, gamma, beta, w1, w2, dout))
    m, c = x.shape
    f = w2.shape[0]
    gq, sq, s2 = np.zeros((c, 2 * f)), np.zeros(2 * f), np.zeros((f, c))
    gr, sr, r2 = np.zeros((c, 2 * f)), np.zeros(2 * f), np.zeros((f, c))
    w1sq = w1 ** 2
    for r in _blocks(m, None):
        xhat, o1, _, _ = _ln(x[r], gamma, beta, eps)
        h = o1 @ w1
        a, b = h[:, :f], h[:, f:]
        dlt = 2.0 ** -9 * np.sqrt((o1 ** 2) @ w1sq)
        ea, eb = dlt[:, :f], dlt[:, f:]
        sg = _sigmoid(a)
        phi = sg * (1.0 + a * (1.0 - sg))               # d silu / da
        dphi = sg * (1.0 - sg) * (2.0 + a * (1.0 - 2.0 * sg))
        do = dout[r]
        du = do @ w2.T
        dh = np.concatenate([du * b * phi, du * a * sg], axis=1)
        edh = np.concatenate([np.abs(du) * (np.abs(phi) * eb + np.abs(b * dphi) * ea),
                              np.abs(du * phi) * ea], axis=1)
        eu = np.abs(phi * b) * ea + np.abs(a * sg) * eb
        gq += (xhat ** 2).T @ (dh ** 2)
        sq += (dh ** 2).sum(axis=0)
        s2 += ((a * sg * b) ** 2).T @ (do ** 2)
        gr += (xhat ** 2).T @ (edh ** 2)
        sr += (edh ** 2).sum(axis=0)
        r2 += (eu ** 2).T @ (do ** 2)

    def regroup(g2, s_2):
        dw1 = np.abs(gamma)[:, None] * np.sqrt(g2) + np.abs(beta)[:, None] * np.sqrt(s_2)[None, :]
        return dw1, np.sqrt((w1sq * g2).sum(axis=1)), np.sqrt(w1sq @ s_2)

    S1, Sg, Sb = regroup(gq, sq)
    R1, Rg, Rb = regroup(gr, sr)
    return (S1, np.sqrt(s2), Sg, Sb), (R1, np.sqrt(r2), Rg, Rb)

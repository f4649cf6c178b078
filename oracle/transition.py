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

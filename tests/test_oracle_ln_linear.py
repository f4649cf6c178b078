"""Pins for the fused layer-norm + linear oracle (oracle/ln_linear.c).

The oracle follows the paper's table of fused operators (Section IV, fused
layer-norm & linear projection; appendix table).  Each pin checks it against
something other than itself: torch's float64 layer_norm and matmul (a
library routine), torch autograd, central finite differences, invariants of
layer normalisation, and a closed form.
"""
import numpy as np
import pytest
import torch

import oracle

EPS = 1e-5


def rnd(m, k, n, seed):
    r = np.random.default_rng(seed)
    return (r.normal(size=(m, k)) * 2 + 0.5, r.normal(size=k), r.normal(size=k),
            r.normal(size=(k, n)) / np.sqrt(k), r.normal(size=(m, n)))


def torch_ref(x, g, b, w, do, eps=EPS):
    t = [torch.tensor(a, dtype=torch.float64, requires_grad=True) for a in (x, g, b, w)]
    o2 = torch.nn.functional.layer_norm(t[0], [x.shape[1]], t[1], t[2], eps) @ t[3]
    o2.backward(torch.tensor(do, dtype=torch.float64))
    return o2.detach().numpy(), [a.grad.numpy() for a in t]


@pytest.mark.parametrize("m,k,n,seed", [(5, 4, 3, 0), (33, 128, 20, 1), (9, 64, 516, 2)])
def test_forward_and_backward_match_torch(m, k, n, seed):
    x, g, b, w, do = rnd(m, k, n, seed)
    o2, mean, rstd = oracle.lnl_fwd(x, g, b, w, EPS)
    ref, (dx_r, dg_r, db_r, dw_r) = torch_ref(x, g, b, w, do)
    np.testing.assert_allclose(o2, ref, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(mean, x.mean(1), rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(rstd, 1 / np.sqrt(x.var(1) + EPS), rtol=1e-12)
    dx, dw, dg, db = oracle.lnl_bwd(x, g, b, w, do, EPS)
    for got, want in ((dx, dx_r), (dw, dw_r), (dg, dg_r), (db, db_r)):
        np.testing.assert_allclose(got, want, rtol=1e-11, atol=1e-11)


def test_backward_matches_central_finite_differences():
    m, k, n = 3, 5, 4
    x, g, b, w, do = rnd(m, k, n, 7)

    def loss(xx, gg, bb, ww):
        return float(np.sum(do * oracle.lnl_fwd(xx, gg, bb, ww, EPS)[0]))

    dx, dw, dg, db = oracle.lnl_bwd(x, g, b, w, do, EPS)
    h = 1e-6
    for arr, grad, idx in ((x, dx, 0), (g, dg, 1), (b, db, 2), (w, dw, 3)):
        num = np.zeros_like(arr)
        for i in np.ndindex(arr.shape):
            args_p = [x.copy(), g.copy(), b.copy(), w.copy()]
            args_m = [x.copy(), g.copy(), b.copy(), w.copy()]
            args_p[idx][i] += h
            args_m[idx][i] -= h
            num[i] = (loss(*args_p) - loss(*args_m)) / (2 * h)
        np.testing.assert_allclose(grad, num, rtol=1e-6, atol=1e-7)


def test_row_shift_and_scale_invariance():
    # adding a constant to a row, or scaling it (eps = 0), leaves the
    # normalised row and hence o2 unchanged
    x, g, b, w, do = rnd(11, 16, 7, 3)
    c = np.arange(11.0)[:, None] - 4.0
    o2 = oracle.lnl_fwd(x, g, b, w, 0.0)[0]
    np.testing.assert_allclose(oracle.lnl_fwd(x + c, g, b, w, 0.0)[0], o2, rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(oracle.lnl_fwd(x * 3.5, g, b, w, 0.0)[0], o2, rtol=1e-10,
                               atol=1e-10)
    # so the gradient of a row is orthogonal to the constant direction and,
    # with eps = 0, to the row itself
    dx = oracle.lnl_bwd(x, g, b, w, do, 0.0)[0]
    np.testing.assert_allclose(dx.sum(1), 0.0, atol=1e-10)
    np.testing.assert_allclose((dx * x).sum(1), 0.0, atol=1e-9)


def test_zero_gamma_gives_beta_projection_and_no_input_gradient():
    x, g, b, w, do = rnd(6, 8, 5, 4)
    g0 = np.zeros_like(g)
    o2 = oracle.lnl_fwd(x, g0, b, w, EPS)[0]
    np.testing.assert_allclose(o2, np.broadcast_to(b @ w, o2.shape), rtol=1e-13, atol=1e-13)
    dx, dw, dg, db = oracle.lnl_bwd(x, g0, b, w, do, EPS)
    np.testing.assert_allclose(dx, 0.0, atol=1e-15)
    np.testing.assert_allclose(db, (do @ w.T).sum(0), rtol=1e-12)


def test_closed_form_two_features():
    # K = 2: xhat = +-(a - b) / 2 * rstd with rstd = 1 / sqrt(((a - b) / 2)^2 + eps)
    x = np.array([[3.0, 1.0], [-2.0, 5.0]])
    g, b = np.array([2.0, -1.0]), np.array([0.5, 0.25])
    w = np.eye(2)
    o2, mean, rstd = oracle.lnl_fwd(x, g, b, w, EPS)
    half = (x[:, 0] - x[:, 1]) / 2
    r = 1 / np.sqrt(half ** 2 + EPS)
    np.testing.assert_allclose(mean, x.mean(1), rtol=1e-15)
    np.testing.assert_allclose(rstd, r, rtol=1e-14)
    np.testing.assert_allclose(o2[:, 0], half * r * g[0] + b[0], rtol=1e-14)
    np.testing.assert_allclose(o2[:, 1], -half * r * g[1] + b[1], rtol=1e-14)


def test_row_subset_matches_full_run():
    x, g, b, w, do = rnd(20, 32, 9, 5)
    o2 = oracle.lnl_fwd(x, g, b, w, EPS)[0]
    dx = oracle.lnl_bwd(x, g, b, w, do, EPS, sums=False)[0]
    rows = [0, 7, 19]
    o2s = oracle.lnl_fwd(x, g, b, w, EPS, rows=rows)[0]
    dxs = oracle.lnl_bwd(x, g, b, w, do, EPS, rows=rows, sums=False)[0]
    np.testing.assert_array_equal(o2s[rows], o2[rows])
    np.testing.assert_array_equal(dxs[rows], dx[rows])
    assert np.isnan(o2s[1]).all() and np.isnan(dxs[1]).all()

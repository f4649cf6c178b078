"""Pins for the transition-layer oracle (oracle/transition.py).

The oracle follows Section IV (fused SwiGLU, fused transition layer) and the
appendix listing of the transition layer.  Each pin checks it against
something other than itself: torch's float64 layer_norm, silu and matmul
with autograd (library routines), central finite differences, invariants of
layer normalisation and a closed form of the gate.
"""
import numpy as np
import pytest
import torch

from oracle import transition as T

EPS = 1e-5


def rnd(m, c, f, seed):
    r = np.random.default_rng(seed)
    return (r.normal(size=(m, c)) * 1.5 + 0.3, 1 + 0.2 * r.normal(size=c), 0.2 * r.normal(size=c),
            r.normal(size=(c, 2 * f)) / np.sqrt(c), r.normal(size=(f, c)) / np.sqrt(f),
            r.normal(size=(m, c)))


def torch_ref(x, g, b, w1, w2, do, eps=EPS):
    t = [torch.tensor(a, dtype=torch.float64, requires_grad=True) for a in (x, g, b, w1, w2)]
    f = w2.shape[0]
    h = torch.nn.functional.layer_norm(t[0], [x.shape[1]], t[1], t[2], eps) @ t[3]
    out = (torch.nn.functional.silu(h[:, :f]) * h[:, f:]) @ t[4]
    out.backward(torch.tensor(do, dtype=torch.float64))
    return out.detach().numpy(), [a.grad.numpy() for a in t]


@pytest.mark.parametrize("m,c,f,seed", [(5, 4, 3, 0), (37, 128, 64, 1), (20, 16, 512, 2)])
def test_matches_torch_autograd(m, c, f, seed):
    x, g, b, w1, w2, do = rnd(m, c, f, seed)
    out, mean, rstd = T.trn_fwd(x, g, b, w1, w2, EPS)
    ref, (dx_r, dg_r, db_r, dw1_r, dw2_r) = torch_ref(x, g, b, w1, w2, do)
    np.testing.assert_allclose(out, ref, rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(mean, x.mean(1), rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(rstd, 1 / np.sqrt(x.var(1) + EPS), rtol=1e-12)
    dx, dw1, dw2, dg, db = T.trn_bwd(x, g, b, w1, w2, do, EPS)
    for got, want in ((dx, dx_r), (dw1, dw1_r), (dw2, dw2_r), (dg, dg_r), (db, db_r)):
        np.testing.assert_allclose(got, want, rtol=1e-10, atol=1e-10)


def test_backward_matches_central_finite_differences():
    m, c, f = 3, 5, 4
    x, g, b, w1, w2, do = rnd(m, c, f, 7)
    args = [x, g, b, w1, w2]

    def loss(vals):
        return float(np.sum(do * T.trn_fwd(*vals, EPS)[0]))

    grads = T.trn_bwd(x, g, b, w1, w2, do, EPS)
    # trn_bwd returns (dx, dw1, dw2, dgamma, dbeta); args are (x, g, b, w1, w2)
    want = {0: grads[0], 1: grads[3], 2: grads[4], 3: grads[1], 4: grads[2]}
    h = 1e-6
    for i, a in enumerate(args):
        num = np.zeros_like(a)
        for idx in np.ndindex(a.shape):
            p = [v.copy() for v in args]
            p[i][idx] += h
            lp = loss(p)
            p[i][idx] -= 2 * h
            num[idx] = (lp - loss(p)) / (2 * h)
        np.testing.assert_allclose(want[i], num, rtol=1e-6, atol=1e-7)


def test_row_shift_and_scale_invariance():
    x, g, b, w1, w2, do = rnd(6, 32, 16, 3)
    out = T.trn_fwd(x, g, b, w1, w2, 0.0)[0]
    out2 = T.trn_fwd(2.5 * x + 4.0, g, b, w1, w2, 0.0)[0]
    np.testing.assert_allclose(out, out2, rtol=1e-10, atol=1e-10)
    dx = T.trn_bwd(x, g, b, w1, w2, do, 0.0)[0]
    # the output does not change along x -> x + t and x -> (1 + t) x
    np.testing.assert_allclose(dx.sum(1), 0, atol=1e-10)
    np.testing.assert_allclose((dx * x).sum(1), 0, atol=1e-9)


def test_closed_form_constant_rows():
    """gamma = 0 makes o1 = beta for every row: then a = beta W1a and
    b = beta W1b are constants, out = (a sigmoid(a) b) W2 for every row, and
    no gradient reaches x."""
    x, g, b, w1, w2, do = rnd(4, 8, 6, 5)
    g = np.zeros_like(g)
    out = T.trn_fwd(x, g, b, w1, w2, EPS)[0]
    a, bb = b @ w1[:, :6], b @ w1[:, 6:]
    want = (a / (1 + np.exp(-a)) * bb) @ w2
    np.testing.assert_allclose(out, np.broadcast_to(want, out.shape), rtol=1e-12, atol=1e-12)
    dx, dw1, dw2, dg, db = T.trn_bwd(x, g, b, w1, w2, do, EPS)
    np.testing.assert_allclose(dx, 0, atol=1e-12)
    # dW2 = u^T sum(dout) with the constant u
    u = a / (1 + np.exp(-a)) * bb
    np.testing.assert_allclose(dw2, np.outer(u, do.sum(0)), rtol=1e-12, atol=1e-12)


def test_gate_special_values():
    """b-half of W1 chosen so that b = 1 and a = 0 on every row: then
    u = 0 (silu(0) = 0), out = 0, da = du / 2 (silu'(0) = 1/2), db = 0."""
    m, c, f = 3, 4, 2
    x, g, b, w1, w2, do = rnd(m, c, f, 9)
    g = np.zeros(c)
    b = np.zeros(c)
    b[0] = 1.0
    w1 = np.zeros((c, 2 * f))
    w1[0, f:] = 1.0  # b = 1, a = 0
    out = T.trn_fwd(x, g, b, w1, w2, EPS)[0]
    np.testing.assert_allclose(out, 0, atol=1e-15)
    dx, dw1, dw2, dg, db = T.trn_bwd(x, g, b, w1, w2, do, EPS)
    du = do @ w2.T
    # dW1 = o1^T dh with o1 = e_0 for every row
    np.testing.assert_allclose(dw1[0, :f], 0.5 * du.sum(0), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dw1[0, f:], 0, atol=1e-15)
    np.testing.assert_allclose(dw1[1:], 0, atol=1e-15)
    np.testing.assert_allclose(dw2, 0, atol=1e-15)


def test_row_subset_matches_full_run():
    x, g, b, w1, w2, do = rnd(50, 16, 8, 11)
    rows = [0, 7, 49]
    out, mean, rstd = T.trn_fwd(x, g, b, w1, w2, EPS)
    o2, m2, r2 = T.trn_fwd(x, g, b, w1, w2, EPS, rows=rows)
    np.testing.assert_array_equal(o2[rows], out[rows])
    assert np.isnan(o2[1]).all()
    full = T.trn_bwd(x, g, b, w1, w2, do, EPS)
    part = T.trn_bwd(x, g, b, w1, w2, do, EPS, rows=rows, sums=False)
    np.testing.assert_array_equal(part[0][rows], full[0][rows])
    assert part[1] is None
    both = T.trn_bwd(x, g, b, w1, w2, do, EPS, rows=rows)
    for a, bb in zip(both[1:], full[1:]):
        np.testing.assert_allclose(a, bb, rtol=1e-13, atol=1e-13)


# ---- the pins catch plausible slips --------------------------------------------------
# Each case plants one mistake in a temporary copy of oracle/transition.py,
# loads it as a separate module and requires at least one pin to fail.

MUTATIONS = {
    "silu_prime_dropped": ("sg * (1.0 + a * (1.0 - sg))", "sg", 1),
    "db_uses_sigmoid": ("du * silu], axis=1)", "du * sg], axis=1)", 1),
    "halves_swapped": ("a, b = h[:, :f], h[:, f:]", "b, a = h[:, :f], h[:, f:]", 2),
    "dw2_without_b": ("dw2 += (silu * b).T @ do", "dw2 += silu.T @ do", 1),
    "c1_dropped": ("rs[:, None] * (wdy - c1 * xhat - c2)", "rs[:, None] * (wdy - c2)", 1),
    "gamma_missing_in_dx": ("wdy = do1 * gamma", "wdy = do1", 1),
    "unbiased_variance": ("var = ((x - mean[:, None]) ** 2).mean(axis=1)",
                          "var = ((x - mean[:, None]) ** 2).sum(axis=1) / (x.shape[1] - 1)", 1),
    "dw1_uses_xhat": ("dw1 += o1.T @ dh", "dw1 += xhat.T @ dh", 1),
    "out_without_gate": ("out[r] = (a * _sigmoid(a) * b) @ w2", "out[r] = (a * b) @ w2", 1),
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_catch_mutation(name, tmp_path):
    import importlib.util
    import inspect
    old, new, count = MUTATIONS[name]
    src = inspect.getsource(T)
    # every occurrence is mutated (the error-scale helper repeats some steps)
    assert src.count(old) >= count, f"mutation anchor for {name} not found"
    path = tmp_path / "transition_mut.py"
    path.write_text(src.replace(old, new))
    spec = importlib.util.spec_from_file_location("transition_mut", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    pins = [lambda: test_matches_torch_autograd(5, 4, 3, 0),
            test_backward_matches_central_finite_differences,
            test_row_shift_and_scale_invariance, test_closed_form_constant_rows,
            test_gate_special_values]
    failed = 0
    g = globals()
    saved = g["T"]
    g["T"] = mod
    try:
        for p in pins:
            try:
                p()
            except AssertionError:
                failed += 1
    finally:
        g["T"] = saved
    assert failed > 0, f"no pin caught {name}"

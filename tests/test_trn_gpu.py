"""GPU parity of the fused transition layer (through the C ABI) against the
fp64 oracle, on the same seeded bf16 inputs.

Tolerance: the bf16 bound used for the attention, |gpu - oracle| <= 2e-2 +
1e-2 |oracle| elementwise plus a relative Frobenius error <= 1e-2; the fp32
row statistics to 1e-5.  The sums over rows (dW1, dW2, dgamma, dbeta) take
the bound the layer-norm + linear sums use, which depends on the oracle's
values only: the absolute part is 2e-2 times the RMS of the oracle's
entries of that sum (a sum of m terms with relative bf16 rounding errors
grows like the l2 norm of its terms, which is the size of a typical entry).
Small problems are compared in full (several 256-row blocks and 32-row
tiles, ragged tails, one to sixteen 32-column hidden chunks); the N = 768
pair representation (589824 rows) is compared on sampled rows for out and dx
and in full for the sums over rows.
"""
import numpy as np
import pytest
import torch

from oracle import transition as OT
from paper_2506_20686_amd import binding as B
from paper_2506_20686_amd import workloads as W

from test_lnl_gpu import close


def check_sums(got, ref):
    for name, g, r in zip(("dw1", "dw2", "dgamma", "dbeta"), got, ref):
        close(name, g, r, row_sum=True)


pytestmark = pytest.mark.gpu
DEV = "cuda:0"
EPS = 1e-5
NAMES = ("x", "gamma", "beta", "w1", "w2", "dout")


def to_dev(t):
    return {k: t[k].to(DEV) for k in NAMES}


def run(t, bwd=True):
    d = to_dev(t)
    out, mean, rstd = B.transition_fwd(d["x"], d["gamma"], d["beta"], d["w1"], d["w2"], EPS)
    grads = None
    if bwd:
        grads = B.transition_bwd(d["x"], d["gamma"], d["beta"], d["w1"], d["w2"], mean, rstd,
                                 d["dout"])
    torch.cuda.synchronize()
    return out, mean, rstd, grads


SHAPES = [(1, 128), (37, 128), (300, 512), (1000, 256), (257, 384), (2000, 512)]


@pytest.mark.parametrize("m,f", SHAPES)
def test_forward_and_backward_full(m, f):
    t = W.trn_inputs(m, seed=100 + m, f=f)
    print(f"\n[transition m={m} f={f}]", flush=True)
    out, mean, rstd, (dx, dw1, dw2, dg, db) = run(t)
    ro, rmean, rrstd = OT.trn_fwd(t["x"], t["gamma"], t["beta"], t["w1"], t["w2"], EPS)
    close("out", out, ro)
    np.testing.assert_allclose(mean.cpu().numpy(), rmean, rtol=1e-5, atol=1e-5)
    np.testing.assert_allclose(rstd.cpu().numpy(), rrstd, rtol=1e-5, atol=1e-5)
    rdx, rdw1, rdw2, rdg, rdb = OT.trn_bwd(t["x"], t["gamma"], t["beta"], t["w1"], t["w2"],
                                           t["dout"], EPS)
    close("dx", dx, rdx)
    check_sums((dw1, dw2, dg, db), (rdw1, rdw2, rdg, rdb))


def test_pair_transition_n768():
    """The N = 768 pair representation in the benchmark's launch
    configuration: out and dx on sampled rows, the sums over rows in full."""
    m = 768 * 768
    t = W.trn_inputs(m, seed=0)
    print(f"\n[transition m={m} f={W.TRN_F}]", flush=True)
    out, mean, rstd, (dx, dw1, dw2, dg, db) = run(t)
    rows = sorted({0, 1, 31, 32, 255, 256, 4095, m // 2, m - 33, m - 1})
    ro, rmean, rrstd = OT.trn_fwd(t["x"], t["gamma"], t["beta"], t["w1"], t["w2"], EPS,
                                  rows=rows)
    close("out", out.cpu()[rows], ro[rows])
    np.testing.assert_allclose(mean.cpu().numpy()[rows], rmean[rows], rtol=1e-5, atol=1e-5)
    np.testing.assert_allclose(rstd.cpu().numpy()[rows], rrstd[rows], rtol=1e-5, atol=1e-5)
    rdx, rdw1, rdw2, rdg, rdb = OT.trn_bwd(t["x"], t["gamma"], t["beta"], t["w1"], t["w2"],
                                           t["dout"], EPS, rows=rows)
    close("dx", dx.cpu()[rows], rdx[rows])
    check_sums((dw1, dw2, dg, db), (rdw1, rdw2, rdg, rdb))


def test_transition_is_bitwise_deterministic():
    t = W.trn_inputs(5000, seed=4)
    a = run(t)
    b = run(t)
    for x, y in zip(a[:3], b[:3]):
        assert torch.equal(x, y)
    for x, y in zip(a[3], b[3]):
        assert torch.equal(x, y)

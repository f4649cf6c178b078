"""GPU parity of the starting node over a range of rows (one GPU's share of
the row-sharded pair map, Section IV-B) against the fp64 oracle, and its
consistency with the whole-map call.

The range's rows are independent attention problems, so its out, lse, dq,
dk, dv and dg are compared with the oracle's rows r0 .. r0 + rows - 1 of the
whole map, to the same bounds as the whole call (fp32: 1e-4 absolute; bf16:
2e-2 + 1e-2 |ref| elementwise and 1e-2 relative Frobenius).  The range's
fp32 bias-gradient term is the oracle's bias gradient with dout set to zero
outside the range (rows with zero dout contribute nothing to it).  The same
rows of a whole-map call run the same arithmetic, so they must agree
bitwise; the terms of ranges that cover the map must add up to the whole
call's bias gradient.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2506_20686_amd import binding as B
from paper_2506_20686_amd import workloads as W

from test_parity_gpu import DEV, close, inputs, to_dev

pytestmark = pytest.mark.gpu


def run_rows(t, r0, rows, scale=None):
    sl = slice(r0, r0 + rows)
    d = {k: t[k][sl].contiguous().to(DEV) for k in ("q", "k", "v", "g", "dout")}
    m = None if t.get("mask") is None else t["mask"][sl].contiguous().to(DEV)
    bias = t["bias"].to(DEV)
    out, lse = B.rows_fwd(d["q"], d["k"], d["v"], d["g"], bias, m, scale)
    grads = B.rows_bwd(d["q"], d["k"], d["v"], d["g"], bias, out, lse, d["dout"], m, scale)
    torch.cuda.synchronize()
    return out, lse, grads


def zero_outside(dout, r0, rows):
    z = torch.zeros_like(dout)
    z[r0:r0 + rows] = dout[r0:r0 + rows]
    return z


def check_range(t, r0, rows, dtype, scale=None, db_queries=None):
    out, lse, grads = run_rows(t, r0, rows, scale)
    rl = list(range(r0, r0 + rows))
    ro, rlse = oracle.fwd(B.STARTING, t["q"], t["k"], t["v"], t["g"], t["bias"], t.get("mask"),
                          scale, rows=rl)
    rg = oracle.bwd(B.STARTING, t["q"], t["k"], t["v"], t["g"], t["bias"],
                    zero_outside(t["dout"], r0, rows), t.get("mask"), scale, rows=rl,
                    db_queries=db_queries)
    close("out", out, ro[r0:r0 + rows], dtype)
    close("lse", lse, rlse[r0:r0 + rows], dtype)
    for name, a, b in zip(("dq", "dk", "dv", "dg"), grads[:4], rg[:4]):
        close(name, a, b[r0:r0 + rows], dtype)
    assert grads[4].dtype == torch.float32
    sel = None if db_queries is None else (sorted(db_queries),)
    close("dbias_partial", grads[4], rg[4], dtype, sel)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("n,h,r0,rows,mask_kind", [
    (1, 1, 0, 1, "none"), (37, 2, 0, 37, "random"), (37, 2, 36, 1, "random"),
    (100, 4, 50, 13, "pair"), (130, 1, 3, 70, "random"), (96, 3, 24, 24, "none"),
])
def test_range_full(dtype, n, h, r0, rows, mask_kind):
    t = inputs(n, h, dtype, seed=3000 + n + 11 * r0 + rows, mask_kind=mask_kind)
    print(f"\n[rows n={n} h={h} r0={r0} rows={rows} {dtype}]", flush=True)
    check_range(t, r0, rows, dtype)


def test_range_degenerate_mask():
    n, h = 40, 2
    t = inputs(n, h, torch.bfloat16, seed=78, mask_kind="none")
    m = torch.ones(n, n, dtype=torch.uint8)
    m[10:20] = 0  # rows with no valid key: out 0, lse -inf, no gradient
    t["mask"] = m
    check_range(t, 8, 16, torch.bfloat16)


def test_ranges_agree_with_whole_call():
    t = inputs(100, 4, torch.bfloat16, seed=91, mask_kind="random")
    d = to_dev(t)
    out, lse = B.fwd(d["q"], d["k"], d["v"], d["g"], d["bias"], d["mask"], B.STARTING)
    grads = B.bwd(d["q"], d["k"], d["v"], d["g"], d["bias"], out, lse, d["dout"], d["mask"],
                  B.STARTING)
    db_sum = torch.zeros(t["bias"].shape, dtype=torch.float32, device=DEV)
    for r0, rows in ((0, 33), (33, 1), (34, 64), (98, 2)):
        o, l, g = run_rows(t, r0, rows)
        sl = slice(r0, r0 + rows)
        # the same rows run the same arithmetic: bitwise equal
        assert torch.equal(o, out[sl]) and torch.equal(l, lse[sl])
        for a, b in zip(g[:4], grads[:4]):
            assert torch.equal(a, b[sl])
        db_sum += g[4]
    # the terms add up to the whole gradient (different summation order:
    # equal to the whole call's rounding)
    ref = oracle.bwd(B.STARTING, t["q"], t["k"], t["v"], t["g"], t["bias"], t["dout"],
                     t["mask"])[4]
    close("sum of dbias terms", db_sum, ref, torch.bfloat16)
    # rounded to bf16, the summed terms and the whole call's gradient differ
    # by at most one bf16 unit (2^-7 relative) where their fp32 sums differ
    a, b = db_sum.to(torch.bfloat16).float(), grads[4].float()
    assert torch.all((a - b).abs() <= 2.0 ** -7 * torch.maximum(a.abs(), b.abs()))


def test_range_is_bitwise_deterministic():
    rw = W.ROWS_WORKLOADS["tri_rows_bf16_n768_r96"]
    s = W.rows_inputs(rw)
    d = {k: v.to(DEV) for k, v in s.items() if k != "whole"}
    r1 = B.rows_fwd(d["q"], d["k"], d["v"], d["g"], d["bias"], d["mask"])
    r2 = B.rows_fwd(d["q"], d["k"], d["v"], d["g"], d["bias"], d["mask"])
    assert all(torch.equal(a, b) for a, b in zip(r1, r2))
    g1 = B.rows_bwd(d["q"], d["k"], d["v"], d["g"], d["bias"], *r1, d["dout"], d["mask"])
    g2 = B.rows_bwd(d["q"], d["k"], d["v"], d["g"], d["bias"], *r1, d["dout"], d["mask"])
    assert all(torch.equal(a, b) for a, b in zip(g1, g2))


def test_shard_workload_sampled():
    """One GPU's 96 rows of the N = 768 map, in the benchmark's launch
    configuration, on sampled rows and bias-gradient queries."""
    rw = W.ROWS_WORKLOADS["tri_rows_bf16_n768_r96"]
    s = W.rows_inputs(rw)
    t = s["whole"]
    print(f"\n[{rw.name}]", flush=True)
    out, lse, grads = run_rows(t, rw.r0, rw.rows)
    local = sorted({0, 1, 47, rw.rows - 1})
    rl = [rw.r0 + i for i in local]
    qs = sorted({0, 255, 767})
    ro, rlse = oracle.fwd(B.STARTING, t["q"], t["k"], t["v"], t["g"], t["bias"], t["mask"],
                          rows=rl)
    rg = oracle.bwd(B.STARTING, t["q"], t["k"], t["v"], t["g"], t["bias"],
                    zero_outside(t["dout"], rw.r0, rw.rows), t["mask"], rows=rl, db_queries=qs)
    dt = torch.bfloat16
    close("out", out[local], ro[rl], dt)
    close("lse", lse[local], rlse[rl], dt)
    for name, a, b in zip(("dq", "dk", "dv", "dg"), grads[:4], rg[:4]):
        close(name, a[local], b[rl], dt)
    close("dbias_partial", grads[4], rg[4], dt, (qs,))

"""GPU parity of triangle attention with head dimension d = 64 against the
fp64 oracle, with the tolerances of the d = 32 tests, including a batched
call and the run-to-run determinism.  bf16 runs the DMA kernels' 64-channel
variants (positions staged as two 32-channel halves), fp32 the
register-staged kernels instantiated for 64 channels.  The benchmark's
d = 64 workload (N = 768) is checked on sampled rows and a whole 128-query
block of the bias gradient."""
import pytest
import torch

import oracle
from paper_2506_20686_amd import binding as B
from paper_2506_20686_amd import workloads as W

from test_parity_gpu import DEV, close

pytestmark = pytest.mark.gpu


def inputs64(n, h, dtype, seed, mask_kind="random"):
    t, gen = W.make_inputs(n, h, 64, dtype, seed=seed)
    if mask_kind == "random":
        t["mask"] = W.random_mask(n, 0.8, gen)
    elif mask_kind == "pair":
        t["mask"] = W.pair_mask(n, max(1, n // 6))
    else:
        t["mask"] = None
    return t


def check(t, node, dtype, rows=None, db_queries=None):
    d = {k: (v.to(DEV) if isinstance(v, torch.Tensor) else v) for k, v in t.items()}
    out, lse = B.fwd(d["q"], d["k"], d["v"], d["g"], d["bias"], d["mask"], node)
    grads = B.bwd(d["q"], d["k"], d["v"], d["g"], d["bias"], out, lse, d["dout"], d["mask"], node)
    torch.cuda.synchronize()
    ro, rl = oracle.fwd(node, t["q"], t["k"], t["v"], t["g"], t["bias"], t["mask"], rows=rows)
    rg = oracle.bwd(node, t["q"], t["k"], t["v"], t["g"], t["bias"], t["dout"], t["mask"],
                    rows=rows, db_queries=db_queries)
    sel = None
    if rows is not None:
        sel = (rows,) if node == B.STARTING else (slice(None), rows)
    close("out", out, ro, dtype, sel)
    close("lse", lse, rl, dtype, sel)
    for name, a, r in zip(("dq", "dk", "dv", "dg"), grads[:4], rg[:4]):
        close(name, a, r, dtype, sel)
    bsel = None
    if db_queries is not None:
        bsel = (db_queries,) if node == B.STARTING else (slice(None), db_queries)
    close("dbias", grads[4], rg[4], dtype, bsel)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("node", [B.STARTING, B.ENDING])
@pytest.mark.parametrize("n,h,mask_kind", [(1, 1, "none"), (37, 2, "random"), (100, 3, "pair"),
                                           (130, 1, "random")])
def test_d64_full(dtype, node, n, h, mask_kind):
    print(f"\n[d64 n={n} h={h} node={node} {dtype}]", flush=True)
    check(inputs64(n, h, dtype, seed=800 + n + node, mask_kind=mask_kind), node, dtype)


@pytest.mark.parametrize("node", [B.STARTING, B.ENDING])
def test_d64_n384_sampled(node):
    n = 384
    t = inputs64(n, 4, torch.bfloat16, seed=71 + node, mask_kind="pair")
    print(f"\n[d64 n={n} node={node}]", flush=True)
    check(t, node, torch.bfloat16, rows=[0, 1, 191, n - 1], db_queries=[0, 200, n - 1])


def test_d64_batched_and_deterministic():
    b, n, h = 2, 60, 2
    parts = [inputs64(n, h, torch.bfloat16, seed=60 + i) for i in range(b)]
    t = {k: torch.stack([p[k] for p in parts]) for k in parts[0]}
    d = {k: v.to(DEV) for k, v in t.items()}
    out, lse = B.fwd(d["q"], d["k"], d["v"], d["g"], d["bias"], d["mask"], B.STARTING)
    grads = B.bwd(d["q"], d["k"], d["v"], d["g"], d["bias"], out, lse, d["dout"], d["mask"],
                  B.STARTING)
    out2, lse2 = B.fwd(d["q"], d["k"], d["v"], d["g"], d["bias"], d["mask"], B.STARTING)
    grads2 = B.bwd(d["q"], d["k"], d["v"], d["g"], d["bias"], out2, lse2, d["dout"], d["mask"],
                   B.STARTING)
    torch.cuda.synchronize()
    assert torch.equal(out, out2) and torch.equal(lse, lse2)
    for a, c in zip(grads, grads2):
        assert torch.equal(a, c)
    for i in range(b):
        ro, rl = oracle.fwd(B.STARTING, t["q"][i], t["k"][i], t["v"][i], t["g"][i], t["bias"][i],
                            t["mask"][i])
        rg = oracle.bwd(B.STARTING, t["q"][i], t["k"][i], t["v"][i], t["g"][i], t["bias"][i],
                        t["dout"][i], t["mask"][i])
        close(f"out[{i}]", out[i], ro, torch.bfloat16)
        for name, a, r in zip(("dq", "dk", "dv", "dg", "dbias"), grads, rg):
            close(f"{name}[{i}]", a[i], r, torch.bfloat16)


@pytest.mark.parametrize("node", [B.STARTING, B.ENDING])
def test_d64_workload_sampled(node):
    """The N = 768, h = 4, d = 64 benchmark workload in its launch configuration."""
    w = W.WORKLOADS["tri_bf16_n768_d64"]
    t = W.workload_inputs(w, node)
    n = w.n
    print(f"\n[d64 workload n={n} node={node}]", flush=True)
    check(t, node, w.dtype, rows=[0, 1, 31, 32, n // 2, n - 1], db_queries=list(range(128, 256)))


@pytest.mark.parametrize("node", [B.STARTING, B.ENDING])
def test_d64_minus_inf_bias_tile(node):
    """An additive -inf bias on every key of the first 32-key tile of one
    query (the other queries of its wave see finite logits there) with 64
    channels per head: the -inf query's weights stay exactly 0."""
    n, h, q0 = 70, 2, 5
    t = inputs64(n, h, torch.bfloat16, seed=4343 + node, mask_kind="none")
    bias = t["bias"].clone()
    if node == B.STARTING:
        bias[q0, :32, :] = float("-inf")  # bias[q][k][h]
    else:
        bias[:32, q0, :] = float("-inf")  # the ending node reads bias[k][i][h]
    t["bias"] = bias
    check(t, node, torch.bfloat16)

"""GPU parity of triangle attention with head dimension d = 16 against the
fp64 oracle (d = 16), with the tolerances of the d = 32 tests.  bf16 d = 16
runs the DMA kernels on the 16-channel tensors directly (the second
16-channel step of every contraction over channels is skipped, channels
16..31 are never stored); fp32 d = 16 runs the d = 32 kernels on copies whose
channels 16..31 are zero.  Either way the results must equal, bitwise, those
of a d = 32 call on zero-padded inputs: a skipped product of zeros adds exact
zeros.  The benchmark's d = 16 workload (N = 768) is checked on sampled rows
and a whole 128-query block of the bias gradient."""
import pytest
import torch

import oracle
from paper_2506_20686_amd import binding as B
from paper_2506_20686_amd import workloads as W

from test_parity_gpu import DEV, close

pytestmark = pytest.mark.gpu


def inputs16(n, h, dtype, seed, masked=True):
    t, gen = W.make_inputs(n, h, 16, dtype, seed=seed)
    t["mask"] = W.random_mask(n, 0.8, gen) if masked else None
    return t


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("node", [B.STARTING, B.ENDING])
@pytest.mark.parametrize("n,h", [(1, 1), (37, 2), (100, 4)])
def test_d16_matches_oracle(dtype, node, n, h):
    t = inputs16(n, h, dtype, seed=700 + n + node)
    d = {k: (v.to(DEV) if v is not None else None) for k, v in t.items()}
    out, lse = B.fwd(d["q"], d["k"], d["v"], d["g"], d["bias"], d["mask"], node)
    grads = B.bwd(d["q"], d["k"], d["v"], d["g"], d["bias"], out, lse, d["dout"], d["mask"], node)
    torch.cuda.synchronize()
    assert out.shape == (n, n, h, 16)
    ro, rl = oracle.fwd(node, t["q"], t["k"], t["v"], t["g"], t["bias"], t["mask"])
    rg = oracle.bwd(node, t["q"], t["k"], t["v"], t["g"], t["bias"], t["dout"], t["mask"])
    close("out", out, ro, dtype)
    close("lse", lse, rl, dtype)
    for name, a, r in zip(("dq", "dk", "dv", "dg", "dbias"), grads, rg):
        close(name, a, r, dtype)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("node", [B.STARTING, B.ENDING])
def test_d16_equals_padded_d32_bitwise(node, dtype):
    n, h = 64, 2
    t = inputs16(n, h, dtype, seed=31 + node)
    d = {k: v.to(DEV) for k, v in t.items()}

    def pad(x):
        return torch.nn.functional.pad(x, (0, 16)).contiguous()

    scale = 0.25  # 1 / sqrt(16), passed to both calls
    out, lse = B.fwd(d["q"], d["k"], d["v"], d["g"], d["bias"], d["mask"], node, scale)
    grads = B.bwd(d["q"], d["k"], d["v"], d["g"], d["bias"], out, lse, d["dout"], d["mask"],
                  node, scale)
    p = {k: pad(d[k]) for k in ("q", "k", "v", "g", "dout")}
    o2, l2 = B.fwd(p["q"], p["k"], p["v"], p["g"], d["bias"], d["mask"], node, scale)
    g2 = B.bwd(p["q"], p["k"], p["v"], p["g"], d["bias"], o2, l2, p["dout"], d["mask"], node,
               scale)
    assert torch.equal(out, o2[..., :16]) and torch.equal(lse, l2)
    for a, b in zip(grads[:4], g2[:4]):
        assert torch.equal(a, b[..., :16])
    assert torch.equal(grads[4], g2[4])


def test_d16_batched():
    b, n, h = 2, 50, 2
    parts = [inputs16(n, h, torch.bfloat16, seed=40 + i) for i in range(b)]
    t = {k: torch.stack([p[k] for p in parts]) for k in parts[0]}
    d = {k: v.to(DEV) for k, v in t.items()}
    out, lse = B.fwd(d["q"], d["k"], d["v"], d["g"], d["bias"], d["mask"], B.ENDING)
    grads = B.bwd(d["q"], d["k"], d["v"], d["g"], d["bias"], out, lse, d["dout"], d["mask"],
                  B.ENDING)
    torch.cuda.synchronize()
    for i in range(b):
        ro, rl = oracle.fwd(B.ENDING, t["q"][i], t["k"][i], t["v"][i], t["g"][i], t["bias"][i],
                            t["mask"][i])
        rg = oracle.bwd(B.ENDING, t["q"][i], t["k"][i], t["v"][i], t["g"][i], t["bias"][i],
                        t["dout"][i], t["mask"][i])
        close(f"out[{i}]", out[i], ro, torch.bfloat16)
        for name, a, r in zip(("dq", "dk", "dv", "dg", "dbias"), grads, rg):
            close(f"{name}[{i}]", a[i], r, torch.bfloat16)


@pytest.mark.parametrize("node", [B.STARTING, B.ENDING])
def test_d16_workload_sampled(node):
    """The N = 768, h = 4, d = 16 benchmark workload in its launch
    configuration: sampled rows of every output and a 128-query block of the
    bias gradient."""
    w = W.WORKLOADS["tri_bf16_n768_d16"]
    t = W.workload_inputs(w, node)
    n = w.n
    print(f"\n[d16 workload n={n} node={node}]", flush=True)
    d = {k: (v.to(DEV) if isinstance(v, torch.Tensor) else v) for k, v in t.items()}
    out, lse = B.fwd(d["q"], d["k"], d["v"], d["g"], d["bias"], d["mask"], node)
    grads = B.bwd(d["q"], d["k"], d["v"], d["g"], d["bias"], out, lse, d["dout"], d["mask"], node)
    torch.cuda.synchronize()
    rows = [0, 1, 31, 32, n // 2, n - 1]
    qs = list(range(640, 768))
    ro, rl = oracle.fwd(node, t["q"], t["k"], t["v"], t["g"], t["bias"], t["mask"], rows=rows)
    rg = oracle.bwd(node, t["q"], t["k"], t["v"], t["g"], t["bias"], t["dout"], t["mask"],
                    rows=rows, db_queries=qs)
    sel = (rows,) if node == B.STARTING else (slice(None), rows)
    close("out", out, ro, w.dtype, sel)
    close("lse", lse, rl, w.dtype, sel)
    for nm, a, b in zip(("dq", "dk", "dv", "dg"), grads[:4], rg[:4]):
        close(nm, a, b, w.dtype, sel)
    bsel = (qs,) if node == B.STARTING else (slice(None), qs)
    close("dbias", grads[4], rg[4], w.dtype, bsel)


def test_d16_batched_one_launch_equals_per_sample():
    """bf16 d = 16 batches run every kernel once for the batch; each sample
    equals, bitwise, its own unbatched call."""
    b, n, h = 3, 70, 2
    parts = [inputs16(n, h, torch.bfloat16, seed=90 + i) for i in range(b)]
    t = {k: torch.stack([p[k] for p in parts]) for k in parts[0]}
    d = {k: v.to(DEV) for k, v in t.items()}
    for node in (B.STARTING, B.ENDING):
        out, lse = B.fwd(d["q"], d["k"], d["v"], d["g"], d["bias"], d["mask"], node)
        grads = B.bwd(d["q"], d["k"], d["v"], d["g"], d["bias"], out, lse, d["dout"], d["mask"],
                      node)
        for i in range(b):
            o1, l1 = B.fwd(d["q"][i], d["k"][i], d["v"][i], d["g"][i], d["bias"][i],
                           d["mask"][i], node)
            g1 = B.bwd(d["q"][i], d["k"][i], d["v"][i], d["g"][i], d["bias"][i], o1, l1,
                       d["dout"][i], d["mask"][i], node)
            assert torch.equal(out[i], o1) and torch.equal(lse[i], l1)
            for a, c in zip(grads, g1):
                assert torch.equal(a[i], c)


@pytest.mark.parametrize("node", [B.STARTING, B.ENDING])
def test_d16_minus_inf_bias_tile(node):
    """An additive -inf bias on every key of the first 32-key tile of one
    query (the other queries of its wave see finite logits there) with 16
    channels per head: the -inf query's weights stay exactly 0."""
    n, h, q0 = 70, 2, 5
    t = inputs16(n, h, torch.bfloat16, seed=4444 + node, masked=False)
    bias = t["bias"].clone()
    if node == B.STARTING:
        bias[q0, :32, :] = float("-inf")  # bias[q][k][h]
    else:
        bias[:32, q0, :] = float("-inf")  # the ending node reads bias[k][i][h]
    t["bias"] = bias
    d = {k: (v.to(DEV) if v is not None else None) for k, v in t.items()}
    out, lse = B.fwd(d["q"], d["k"], d["v"], d["g"], d["bias"], d["mask"], node)
    grads = B.bwd(d["q"], d["k"], d["v"], d["g"], d["bias"], out, lse, d["dout"], d["mask"], node)
    torch.cuda.synchronize()
    ro, rl = oracle.fwd(node, t["q"], t["k"], t["v"], t["g"], t["bias"], t["mask"])
    rg = oracle.bwd(node, t["q"], t["k"], t["v"], t["g"], t["bias"], t["dout"], t["mask"])
    close("out", out, ro, torch.bfloat16)
    close("lse", lse, rl, torch.bfloat16)
    for name, a, r in zip(("dq", "dk", "dv", "dg", "dbias"), grads, rg):
        close(name, a, r, torch.bfloat16)

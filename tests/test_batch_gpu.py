"""GPU parity of the batched triangle attention (a leading batch axis, a
bias and a mask per sample) against the fp64 oracle run per sample, with the
tolerances of the unbatched tests; bitwise equality of each sample with the
unbatched call on its slices; and bitwise equality of the one-launch batch
(a workspace per sample) with the sample-by-sample run (one shared
workspace)."""
import pytest
import torch

import oracle
from paper_2506_20686_amd import binding as B
from paper_2506_20686_amd import workloads as W

from test_parity_gpu import DEV, close

pytestmark = pytest.mark.gpu


def batch_inputs(b, n, h, dtype, seed):
    parts = []
    for i in range(b):
        t, gen = W.make_inputs(n, h, 32, dtype, seed=seed + i)
        # a different key-validity pattern per sample: random, padded, none valid in a row
        if i % 3 == 0:
            t["mask"] = W.random_mask(n, 0.8, gen)
        elif i % 3 == 1:
            t["mask"] = W.pair_mask(n, max(1, n // 5))
        else:
            m = torch.ones(n, n, dtype=torch.uint8)
            m[n // 2] = 0
            t["mask"] = m
        parts.append(t)
    return {k: torch.stack([p[k] for p in parts]) for k in parts[0]}


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("node", [B.STARTING, B.ENDING])
def test_batched_matches_oracle_per_sample(dtype, node):
    b, n, h = 3, 45, 2
    t = batch_inputs(b, n, h, dtype, seed=500 + 10 * node)
    d = {k: v.to(DEV) for k, v in t.items()}
    out, lse = B.fwd(d["q"], d["k"], d["v"], d["g"], d["bias"], d["mask"], node)
    grads = B.bwd(d["q"], d["k"], d["v"], d["g"], d["bias"], out, lse, d["dout"], d["mask"],
                  node)
    torch.cuda.synchronize()
    for i in range(b):
        ro, rl = oracle.fwd(node, t["q"][i], t["k"][i], t["v"][i], t["g"][i], t["bias"][i],
                            t["mask"][i])
        rg = oracle.bwd(node, t["q"][i], t["k"][i], t["v"][i], t["g"][i], t["bias"][i],
                        t["dout"][i], t["mask"][i])
        close(f"out[{i}]", out[i], ro, dtype)
        close(f"lse[{i}]", lse[i], rl, dtype)
        for name, a, r in zip(("dq", "dk", "dv", "dg", "dbias"), grads, rg):
            close(f"{name}[{i}]", a[i], r, dtype)


@pytest.mark.parametrize("node", [B.STARTING, B.ENDING])
def test_batched_equals_unbatched_bitwise(node):
    b, n, h = 4, 70, 3
    t = batch_inputs(b, n, h, torch.bfloat16, seed=900 + node)
    d = {k: v.to(DEV) for k, v in t.items()}
    out, lse = B.fwd(d["q"], d["k"], d["v"], d["g"], d["bias"], d["mask"], node)
    grads = B.bwd(d["q"], d["k"], d["v"], d["g"], d["bias"], out, lse, d["dout"], d["mask"],
                  node)
    for i in range(b):
        s = {k: v[i].clone() for k, v in d.items()}  # fresh, aligned allocations
        o1, l1 = B.fwd(s["q"], s["k"], s["v"], s["g"], s["bias"], s["mask"], node)
        g1 = B.bwd(s["q"], s["k"], s["v"], s["g"], s["bias"], o1, l1, s["dout"], s["mask"], node)
        assert torch.equal(o1, out[i]) and torch.equal(l1, lse[i])
        for a, r in zip(g1, grads):
            assert torch.equal(a, r[i])


def run_batched(d, node, ws_kind):
    """fwd + bwd of a batch with the one-launch workspace ("grid") or the
    unbatched one ("seq")."""
    bsz, n, h, dd = d["q"].shape[0], d["q"].shape[1], d["q"].shape[3], d["q"].shape[4]
    dt = B.BF16 if d["q"].dtype == torch.bfloat16 else B.F32
    sizes = {"fwd": (B.tri_attn_fwd_batched_workspace_bytes, B.tri_attn_fwd_workspace_bytes),
             "bwd": (B.tri_attn_bwd_batched_workspace_bytes, B.tri_attn_bwd_workspace_bytes)}
    ws = {}
    for kind, (fb, f1) in sizes.items():
        nbytes = fb(node, dt, bsz, n, h, dd) if ws_kind == "grid" else f1(node, dt, n, h, dd)
        ws[kind] = torch.empty(nbytes, dtype=torch.uint8, device=DEV)
    out, lse = B.fwd(d["q"], d["k"], d["v"], d["g"], d["bias"], d.get("mask"), node,
                     workspace=ws["fwd"])
    grads = B.bwd(d["q"], d["k"], d["v"], d["g"], d["bias"], out, lse, d["dout"], d.get("mask"),
                  node, workspace=ws["bwd"])
    torch.cuda.synchronize()
    return (out, lse) + tuple(grads)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("node", [B.STARTING, B.ENDING])
@pytest.mark.parametrize("head_dim", [32, 64])
def test_one_launch_batch_equals_sample_by_sample(dtype, node, head_dim):
    b, n, h = 3, 67, 2
    parts = []
    for i in range(b):
        t, gen = W.make_inputs(n, h, head_dim, dtype, seed=1300 + 7 * i + node)
        t["mask"] = W.random_mask(n, 0.85, gen) if i != 1 else W.pair_mask(n, 9)
        parts.append(t)
    d = {k: torch.stack([p[k] for p in parts]).to(DEV) for k in parts[0]}
    grid = run_batched(d, node, "grid")
    seq = run_batched(d, node, "seq")
    for name, a, r in zip(("out", "lse", "dq", "dk", "dv", "dg", "dbias"), grid, seq):
        assert torch.equal(a, r), name


@pytest.mark.parametrize("node", [B.STARTING, B.ENDING])
def test_one_launch_batch_benchmark_shape(node):
    """Four N = 384 maps (the batched benchmark shape), no mask: the one-launch
    batch equals the sample-by-sample run bitwise."""
    b, n, h = 4, 384, 4
    parts = [W.make_inputs(n, h, 32, torch.bfloat16, seed=1700 + i)[0] for i in range(b)]
    d = {k: torch.stack([p[k] for p in parts]).to(DEV) for k in parts[0] if k != "mask"}
    grid = run_batched(d, node, "grid")
    seq = run_batched(d, node, "seq")
    for name, a, r in zip(("out", "lse", "dq", "dk", "dv", "dg", "dbias"), grid, seq):
        assert torch.equal(a, r), name

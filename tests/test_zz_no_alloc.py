"""The allocation-free forward (tri_attn_fwd_noalloc, through the C ABI)
against the workspace forward (tri_attn_fwd) on the same inputs: the same
kernels run on the same values, so out and lse agree bit for bit (stronger
than the parity bound).  Two calls in a row, the second on a smaller
problem, share the library's scratch array; then a problem whose workspace
exceeds the array is refused before any launch."""
import ctypes

import pytest
import torch

from paper_2506_20686_amd import binding as B
from paper_2506_20686_amd import workloads as W

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _inputs(n, h, dtype, seed, masked):
    t, gen = W.make_inputs(n, h, 32, dtype, seed=seed)
    t["mask"] = W.random_mask(n, 0.8, gen) if masked else None
    return {k: (v.to(DEV) if isinstance(v, torch.Tensor) else v) for k, v in t.items()}


def _both(t, node):
    ref = B.fwd(t["q"], t["k"], t["v"], t["g"], t["bias"], t["mask"], node)
    got = B.fwd_noalloc(t["q"], t["k"], t["v"], t["g"], t["bias"], t["mask"], node)
    torch.cuda.synchronize()
    return ref, got


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("node", [B.STARTING, B.ENDING])
def test_noalloc_matches_workspace_forward(dtype, node):
    # a large problem first, then a smaller one: the second call reuses the
    # scratch array the first one filled
    for n, h, seed, masked in ((300, 4, 11 + node, True), (70, 2, 12 + node, False)):
        print(f"\n[noalloc dtype={dtype} node={node} n={n} h={h}]", flush=True)
        t = _inputs(n, h, dtype, seed, masked)
        (ro, rl), (go, gl) = _both(t, node)
        assert torch.equal(ro, go), (n, h)
        assert torch.equal(rl, gl), (n, h)


def test_noalloc_headline_size():
    """N = 768, h = 4, d = 32 bf16 (about 9.5 MiB of scratch), then N = 33."""
    for n, seed in ((768, 21), (33, 22)):
        print(f"\n[noalloc headline n={n}]", flush=True)
        t = _inputs(n, 4, torch.bfloat16, seed, False)
        (ro, rl), (go, gl) = _both(t, B.STARTING)
        assert torch.equal(ro, go) and torch.equal(rl, gl), n


def test_noalloc_refuses_problems_beyond_its_scratch():
    n, h = 2048, 4  # bias planes alone need 64 MiB
    ws = B.tri_attn_fwd_workspace_bytes(B.STARTING, B.BF16, n, h, 32)
    assert ws > B.FWD_NOALLOC_SCRATCH_BYTES
    fake = 0x10000  # never touched: the size check comes before any HIP call
    st = B.tri_attn_fwd_noalloc(B.STARTING, B.BF16, n, h, 32, 0.1767767, fake, fake, fake,
                                fake, fake, None, fake, fake, None)
    assert st == B.ERR_TOO_LARGE

"""Seeded synthetic workloads for triangle attention.

This module only draws random numbers and builds masks; it holds none of the
method's arithmetic.  The GPU tests, the benchmark and the oracle tests all
take their inputs from here, so both sides see bit-identical values.

Recipe (the same for every workload): one CPU generator seeded with `seed`;
tensors drawn in the order Q, K, V, G, B, dO as float32 standard normals
scaled by their standard deviation, then rounded to the compute dtype (round
to nearest even).  Randomness a workload needs beyond that (a random padding
length) is drawn from the same generator afterwards.

Masks are key masks: a padded token t (t >= n - n_pad) is never attended to
as a key.  For the starting node the key index is the second pair axis
(mask[a][b] = m[b]); for the ending node it is the first (mask[a][b] = m[a]).
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import torch

STARTING, ENDING = 0, 1
NODE_NAMES = {STARTING: "starting", ENDING: "ending"}


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    n: int
    h: int
    d: int
    dtype: torch.dtype
    nodes: tuple
    bias_std: float = 1.0
    pad_frac: float = 0.0        # fixed key padding: floor(pad_frac * n) tokens
    rand_pad_frac: float = 0.0   # random key padding: Uniform{0..floor(rand_pad_frac * n)}
    seed: int = 0
    batch: int = 1               # independent pair maps (sample i drawn with seed + i)

    @property
    def flops_fwd_bwd(self) -> float:
        """Nominal fwd+bwd flop: 4 N^3 H d forward (Q K^T, P V) plus
        10 N^3 H d backward (S recompute, dV, dP, dK, dQ), per sample."""
        return 14.0 * self.batch * self.n ** 3 * self.h * self.d


# Triangle-attention shapes of AF3 pair stacks: H = 4 heads of d = 32.
WORKLOADS = {
    "tri_start_fp32_n32": Workload("tri_start_fp32_n32", 32, 4, 32, torch.float32, (STARTING,)),
    "tri_start_bf16_n256_pad10": Workload("tri_start_bf16_n256_pad10", 256, 4, 32, torch.bfloat16,
                                          (STARTING,), pad_frac=0.10),
    "tri_end_bf16_n384_randpad15": Workload("tri_end_bf16_n384_randpad15", 384, 4, 32,
                                            torch.bfloat16, (ENDING,), rand_pad_frac=0.15),
    "tri_bf16_n768": Workload("tri_bf16_n768", 768, 4, 32, torch.bfloat16, (STARTING, ENDING),
                              bias_std=math.sqrt(2.0)),
    "tri_start_bf16_n1536_pad5": Workload("tri_start_bf16_n1536_pad5", 1536, 4, 32, torch.bfloat16,
                                          (STARTING,), pad_frac=0.05),
    # a batch of four N = 384 maps (per-sample bias and mask) and heads of 16 channels
    "tri_bf16_b4_n384": Workload("tri_bf16_b4_n384", 384, 4, 32, torch.bfloat16, (STARTING, ENDING),
                                 bias_std=math.sqrt(2.0), batch=4),
    "tri_bf16_n768_d16": Workload("tri_bf16_n768_d16", 768, 4, 16, torch.bfloat16,
                                  (STARTING, ENDING), bias_std=math.sqrt(2.0)),
    "tri_bf16_n768_d64": Workload("tri_bf16_n768_d64", 768, 4, 64, torch.bfloat16,
                                  (STARTING, ENDING), bias_std=math.sqrt(2.0)),
}
HEADLINE = "tri_bf16_n768"


@dataclasses.dataclass(frozen=True)
class RowsWorkload:
    """One GPU's share of a row-sharded starting node: rows [r0, r0 + rows)
    of the named whole-map workload (G = n / rows GPUs)."""
    name: str
    base: str
    r0: int
    rows: int

    @property
    def flops_fwd_bwd(self) -> float:
        w = WORKLOADS[self.base]
        return 14.0 * self.rows * w.n ** 2 * w.h * w.d


ROWS_WORKLOADS = {
    # N = 768 split over 8 GPUs: the fourth GPU's 96 rows
    "tri_rows_bf16_n768_r96": RowsWorkload("tri_rows_bf16_n768_r96", "tri_bf16_n768", 288, 96),
}


def rows_inputs(rw: RowsWorkload):
    """The shard's inputs: q, k, v, g, dout, mask [rows, ...] (contiguous
    slices of the whole map's starting-node inputs), the whole bias, plus the
    whole map's inputs under "whole"."""
    t = workload_inputs(WORKLOADS[rw.base], STARTING)
    sl = slice(rw.r0, rw.r0 + rw.rows)
    s = {k: t[k][sl].contiguous() for k in ("q", "k", "v", "g", "dout", "mask")}
    s["bias"] = t["bias"]
    s["whole"] = t
    return s


def key_mask(n: int, n_pad: int, node: int) -> torch.Tensor:
    """[n, n] uint8 mask that excludes the last n_pad tokens as keys."""
    m = (torch.arange(n) < n - n_pad).to(torch.uint8)
    if node == STARTING:
        return m[None, :].expand(n, n).contiguous()
    return m[:, None].expand(n, n).contiguous()


def pair_mask(n: int, n_pad: int) -> torch.Tensor:
    """Token-pair mask m[a] * m[b]: padded rows then have no valid key."""
    m = (torch.arange(n) < n - n_pad).to(torch.uint8)
    return (m[:, None] * m[None, :]).contiguous()


def random_mask(n: int, p_valid: float, gen: torch.Generator) -> torch.Tensor:
    return (torch.rand((n, n), generator=gen) < p_valid).to(torch.uint8)


def make_inputs(n: int, h: int, d: int, dtype: torch.dtype, seed: int = 0,
                bias_std: float = 1.0, std: float = 1.0):
    """Q, K, V, G [n,n,h,d], B [n,n,h], dO [n,n,h,d] on the CPU, plus the
    generator (positioned after dO) for any further draws."""
    gen = torch.Generator("cpu").manual_seed(seed)

    def draw(shape, s):
        return (torch.randn(shape, generator=gen, dtype=torch.float32) * s).to(dtype)

    q = draw((n, n, h, d), std)
    k = draw((n, n, h, d), std)
    v = draw((n, n, h, d), std)
    g = draw((n, n, h, d), std)
    b = draw((n, n, h), bias_std)
    do = draw((n, n, h, d), std)
    return dict(q=q, k=k, v=v, g=g, bias=b, dout=do), gen


def workload_inputs(w: Workload, node: Optional[int] = None):
    """Inputs of a named workload for one node variant: a dict with q, k, v,
    g, bias, dout, mask (uint8 [n,n]) and n_pad; with batch > 1 every tensor
    has a leading batch axis (sample i from seed + i, the same key padding)."""
    node = w.nodes[0] if node is None else node
    if w.batch > 1:
        parts = [workload_inputs(dataclasses.replace(w, batch=1, seed=w.seed + i), node)
                 for i in range(w.batch)]
        t = {k: torch.stack([p[k] for p in parts]) for k in ("q", "k", "v", "g", "bias", "dout",
                                                             "mask")}
        t["n_pad"] = parts[0]["n_pad"]
        t["node"] = node
        return t
    t, gen = make_inputs(w.n, w.h, w.d, w.dtype, w.seed, w.bias_std)
    n_pad = int(math.floor(w.pad_frac * w.n))
    if w.rand_pad_frac > 0:
        hi = int(math.floor(w.rand_pad_frac * w.n))
        n_pad = int(torch.randint(0, hi + 1, (1,), generator=gen).item())
    t["mask"] = key_mask(w.n, n_pad, node)
    t["n_pad"] = n_pad
    t["node"] = node
    return t


# ---- fused layer-norm + linear projection ------------------------------------------------

# The attention's input projection of an AF3 pair stack: the pair
# representation [n*n][c_z = 128] is normalised and projected to Q, K, V, G
# (h*d = 128 columns each) and the bias logits (h = 4 columns).
LNL_K = 128
LNL_COLS = (128, 128, 128, 128, 4)


def lnl_inputs(m: int, cols=LNL_COLS, seed: int = 0, k: int = LNL_K):
    """x [m, k] ~ N(0.3, 1.5^2); gamma ~ 1 + 0.2 N(0, 1); beta ~ 0.2 N(0, 1);
    W [k, sum(cols)] ~ N(0, 1/k); do2 [m, sum(cols)] ~ N(0, 1); drawn in that
    order from one CPU generator, rounded to bf16."""
    gen = torch.Generator("cpu").manual_seed(seed)
    ncols = int(sum(cols))

    def draw(shape, std=1.0, mean=0.0):
        return (torch.randn(*shape, generator=gen) * std + mean).to(torch.bfloat16)

    x = draw((m, k), 1.5, 0.3)
    gamma = draw((k,), 0.2, 1.0)
    beta = draw((k,), 0.2)
    w = draw((k, ncols), 1.0 / math.sqrt(k))
    do2 = draw((m, ncols))
    return dict(x=x, gamma=gamma, beta=beta, w=w, do2=do2, cols=tuple(cols))


# The fused projection's benchmark shape: the attention inputs of the N = 768
# pair representation (m = N^2 rows), and a small case for parity runs.
LNL_WORKLOADS = {
    "lnl_bf16_n768": dict(m=768 * 768, cols=LNL_COLS),
    "lnl_bf16_n64": dict(m=64 * 64, cols=LNL_COLS),
}


def lnl_step_bytes(m: int, cols=LNL_COLS, k: int = LNL_K) -> dict:
    """Algorithmic HBM bytes of one forward + backward of the fused projection
    (each input read once, each output written once; bf16 tensors, fp32
    statistics and weight gradients)."""
    n = int(sum(cols))
    fwd = m * k * 2 + m * n * 2 + m * 8 + k * n * 2 + 4 * k
    bwd = m * k * 2 + m * n * 2 + m * 8 + m * k * 2 + k * n * (2 + 4) + 4 * k + 8 * k
    return {"fwd": fwd, "bwd": bwd}


# ---- transition layer ------------------------------------------------------------------

# The pair transition of an AF3 pair stack: c_z = 128 features, SwiGLU hidden
# width F = 4 c_z = 512 (W1 [128][1024], W2 [512][128]).
TRN_C = 128
TRN_F = 512


def trn_inputs(m: int, seed: int = 0, c: int = TRN_C, f: int = TRN_F):
    """x [m, c] ~ N(0.3, 1.5^2); gamma ~ 1 + 0.2 N(0, 1); beta ~ 0.2 N(0, 1);
    W1 [c, 2f] ~ N(0, 1/c); W2 [f, c] ~ N(0, 1/f); dout [m, c] ~ N(0, 1);
    drawn in that order from one CPU generator, rounded to bf16."""
    gen = torch.Generator("cpu").manual_seed(seed)

    def draw(shape, std=1.0, mean=0.0):
        return (torch.randn(*shape, generator=gen) * std + mean).to(torch.bfloat16)

    x = draw((m, c), 1.5, 0.3)
    gamma = draw((c,), 0.2, 1.0)
    beta = draw((c,), 0.2)
    w1 = draw((c, 2 * f), 1.0 / math.sqrt(c))
    w2 = draw((f, c), 1.0 / math.sqrt(f))
    dout = draw((m, c))
    return dict(x=x, gamma=gamma, beta=beta, w1=w1, w2=w2, dout=dout)


# The benchmark shape: the pair representation of the N = 768 map.
TRN_WORKLOADS = {"trn_bf16_n768": 768 * 768, "trn_bf16_n64": 64 * 64}


def trn_step_flops(m: int, c: int = TRN_C, f: int = TRN_F) -> float:
    """Algorithmic flop of one forward + backward: forward o1 W1 (2 m c 2f) and
    u W2 (2 m f c); backward du (2 m c f), dW2 (2 m f c), dW1 (2 m c 2f) and
    do1 (2 m 2f c): 18 m c f in all (the backward's recomputation of o1 W1 is
    not counted)."""
    return 18.0 * m * c * f

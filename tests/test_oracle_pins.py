"""Pins of the fp64 oracle against things other than itself.

The paper prints no worked numeric example, so the oracle is pinned by
  - a library routine: torch's scaled_dot_product_attention (float64, CPU)
    and its autograd, per (row, head), for O, LSE and every gradient;
  - central finite differences of L = sum(dO * O) for every input;
  - closed forms (zero queries, constant bias, a single valid key, N = 1,
    constant values) and invariants (softmax shift, masked keys, dS row sums);
  - the ending node equal to the transposed starting node;
  - hand-derived rational fixtures (tests/golden/hand_n2.json).
Each pin is chosen so that a plausible slip (a dropped bias, the bias
transposed, a wrong sign, a swapped axis in the ending node, a missing gate
or scale) fails at least one of them.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from paper_2506_20686_amd import workloads as W

pytestmark = pytest.mark.filterwarnings("ignore")
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
STARTING, ENDING = 0, 1


def rnd(n, h, d, seed, bias_std=1.0):
    t, gen = W.make_inputs(n, h, d, torch.float64, seed=seed, bias_std=bias_std)
    return {k: v.numpy() for k, v in t.items()}, gen


def T(x):
    """Swap the two pair axes."""
    return np.ascontiguousarray(np.swapaxes(x, 0, 1))


def sdpa_start(t, mask, scale, grads=False):
    """Starting-node attention through torch's SDPA, one call per (row, head):
    row r attends queries Q[r] over keys K[r] with bias B[:, :, h]."""
    n, _, h, d = t["q"].shape
    ts = {k: torch.tensor(t[k], requires_grad=grads) for k in ("q", "k", "v", "g", "bias")}
    outs = []
    for r in range(n):
        heads = []
        for hh in range(h):
            addm = ts["bias"][:, :, hh]
            if mask is not None:
                neg = torch.zeros(n, dtype=torch.float64)
                neg[torch.tensor(mask[r] == 0)] = -math.inf
                addm = addm + neg[None, :]
            a = F.scaled_dot_product_attention(ts["q"][r, :, hh][None], ts["k"][r, :, hh][None],
                                               ts["v"][r, :, hh][None], attn_mask=addm[None],
                                               scale=scale)[0]
            heads.append(torch.sigmoid(ts["g"][r, :, hh]) * a)
        outs.append(torch.stack(heads, 1))
    return torch.stack(outs, 0), ts


def sdpa_lse_start(t, mask, scale):
    """LSE through SDPA's normaliser: append one extra key whose logit is 0
    (zero key, zero bias) and whose value is a unit vector in an extra
    channel.  Its weight w = 1 / (1 + sum exp s) gives LSE = ln((1 - w) / w)."""
    n, _, h, d = t["q"].shape
    lse = np.zeros((n, n, h))
    for r in range(n):
        for hh in range(h):
            q = torch.tensor(t["q"][r, :, hh])
            k = torch.cat([torch.tensor(t["k"][r, :, hh]), torch.zeros(1, d, dtype=torch.float64)])
            v = torch.zeros(n + 1, 1, dtype=torch.float64)
            v[n, 0] = 1.0
            addm = torch.zeros(n, n + 1, dtype=torch.float64)
            addm[:, :n] = torch.tensor(t["bias"][:, :, hh])
            if mask is not None:
                addm[:, :n][:, torch.tensor(mask[r] == 0)] = -math.inf
            w = F.scaled_dot_product_attention(q[None], k[None], v[None], attn_mask=addm[None],
                                               scale=scale)[0, :, 0]
            lse[r, :, hh] = torch.log((1 - w) / w).numpy()
    return lse


@pytest.mark.parametrize("seed", [1, 2])
def test_forward_matches_sdpa_starting(seed):
    t, gen = rnd(7, 3, 5, seed)
    mask = W.random_mask(7, 0.7, gen).numpy()
    mask[:, 0] = 1  # every row keeps a key, so SDPA is defined everywhere
    scale = 0.37
    out, lse = oracle.fwd(STARTING, t["q"], t["k"], t["v"], t["g"], t["bias"], mask, scale)
    ref, _ = sdpa_start(t, mask, scale)
    np.testing.assert_allclose(out, ref.detach().numpy(), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(lse, sdpa_lse_start(t, mask, scale), rtol=1e-10, atol=1e-11)


@pytest.mark.parametrize("seed", [3, 4])
def test_backward_matches_sdpa_autograd_starting(seed):
    t, gen = rnd(6, 2, 4, seed)
    mask = W.random_mask(6, 0.75, gen).numpy()
    mask[:, 2] = 1
    scale = 0.5
    ref, ts = sdpa_start(t, mask, scale, grads=True)
    (ref * torch.tensor(t["dout"])).sum().backward()
    dq, dk, dv, dg, db = oracle.bwd(STARTING, t["q"], t["k"], t["v"], t["g"], t["bias"],
                                    t["dout"], mask, scale)
    for mine, name in ((dq, "q"), (dk, "k"), (dv, "v"), (dg, "g"), (db, "bias")):
        np.testing.assert_allclose(mine, ts[name].grad.numpy(), rtol=1e-10, atol=1e-12,
                                   err_msg=name)


@pytest.mark.parametrize("node", [STARTING, ENDING])
def test_backward_matches_central_finite_differences(node):
    n, h, d = 4, 2, 3
    t, gen = rnd(n, h, d, 11 + node)
    mask = W.random_mask(n, 0.7, gen).numpy()
    mask[0, :] = 0  # a key (ending) / row (starting) with nothing valid
    mask[1, 1] = 1
    scale = 0.6

    def loss(tt):
        o, _ = oracle.fwd(node, tt["q"], tt["k"], tt["v"], tt["g"], tt["bias"], mask, scale)
        return float((o * t["dout"]).sum())

    grads = dict(zip(("q", "k", "v", "g", "bias"),
                     oracle.bwd(node, t["q"], t["k"], t["v"], t["g"], t["bias"], t["dout"], mask,
                                scale)))
    eps = 1e-6
    for name in ("q", "k", "v", "g", "bias"):
        fd = np.zeros_like(t[name])
        for idx in np.ndindex(t[name].shape):
            tp = dict(t)
            tp[name] = t[name].copy()
            tp[name][idx] += eps
            lp = loss(tp)
            tp[name][idx] -= 2 * eps
            lm = loss(tp)
            fd[idx] = (lp - lm) / (2 * eps)
        np.testing.assert_allclose(grads[name], fd, atol=1e-7, rtol=1e-6, err_msg=name)


@pytest.mark.parametrize("node", [STARTING, ENDING])
def test_ending_is_transposed_starting(node):
    n, h, d = 9, 2, 4
    t, gen = rnd(n, h, d, 21)
    mask = W.random_mask(n, 0.6, gen).numpy()
    scale = 0.3
    other = 1 - node
    o1, l1 = oracle.fwd(node, t["q"], t["k"], t["v"], t["g"], t["bias"], mask, scale)
    tt = {k: T(v) for k, v in t.items()}
    o2, l2 = oracle.fwd(other, tt["q"], tt["k"], tt["v"], tt["g"], tt["bias"], T(mask), scale)
    np.testing.assert_allclose(o1, T(o2), rtol=0, atol=1e-12)
    np.testing.assert_array_equal(np.isinf(l1), np.isinf(T(l2)))
    fin = np.isfinite(l1)
    np.testing.assert_allclose(l1[fin], T(l2)[fin], rtol=0, atol=1e-12)
    g1 = oracle.bwd(node, t["q"], t["k"], t["v"], t["g"], t["bias"], t["dout"], mask, scale)
    g2 = oracle.bwd(other, tt["q"], tt["k"], tt["v"], tt["g"], tt["bias"], tt["dout"], T(mask),
                    scale)
    for a, b in zip(g1, g2):
        np.testing.assert_allclose(a, T(b), rtol=0, atol=1e-12)


def sig(x):
    return 1.0 / (1.0 + np.exp(-x))


@pytest.mark.parametrize("node", [STARTING, ENDING])
def test_closed_forms_zero_query_and_constant_bias(node):
    n, h, d = 6, 2, 3
    t, gen = rnd(n, h, d, 31)
    mask = W.random_mask(n, 0.6, gen).numpy()
    q0 = np.zeros_like(t["q"])
    c = 0.8
    bias = np.full_like(t["bias"], c)
    out, lse = oracle.fwd(node, q0, t["k"], t["v"], t["g"], bias, mask, 0.5)
    for row in range(n):
        keys = [k for k in range(n) if (mask[row, k] if node == STARTING else mask[k, row])]
        for qi in range(n):
            at = (row, qi) if node == STARTING else (qi, row)
            if not keys:
                assert np.all(out[at] == 0) and np.all(lse[at] == -np.inf)
                continue
            vals = [t["v"][(row, k) if node == STARTING else (k, row)] for k in keys]
            np.testing.assert_allclose(out[at], sig(t["g"][at]) * np.mean(vals, 0), atol=1e-13)
            np.testing.assert_allclose(lse[at], c + math.log(len(keys)), atol=1e-13)


@pytest.mark.parametrize("node", [STARTING, ENDING])
def test_closed_form_single_valid_key(node):
    n, h, d = 5, 2, 4
    t, _ = rnd(n, h, d, 41)
    mask = np.zeros((n, n), np.uint8)
    kstar = 3
    if node == STARTING:
        mask[:, kstar] = 1
    else:
        mask[kstar, :] = 1
    scale = 0.7
    out, lse = oracle.fwd(node, t["q"], t["k"], t["v"], t["g"], t["bias"], mask, scale)
    for row in range(n):
        for qi in range(n):
            at = (row, qi) if node == STARTING else (qi, row)
            kat = (row, kstar) if node == STARTING else (kstar, row)
            bat = (qi, kstar) if node == STARTING else (kstar, qi)
            np.testing.assert_allclose(out[at], sig(t["g"][at]) * t["v"][kat], atol=1e-13)
            s = scale * np.sum(t["q"][at] * t["k"][kat], -1) + t["bias"][bat]
            np.testing.assert_allclose(lse[at], s, atol=1e-13)


def test_closed_form_single_token():
    t, _ = rnd(1, 3, 4, 51)
    out, lse = oracle.fwd(STARTING, t["q"], t["k"], t["v"], t["g"], t["bias"], None, 0.25)
    np.testing.assert_allclose(out, sig(t["g"]) * t["v"], atol=1e-14)
    np.testing.assert_allclose(lse, 0.25 * np.sum(t["q"] * t["k"], -1) + t["bias"], atol=1e-14)
    g = oracle.bwd(STARTING, t["q"], t["k"], t["v"], t["g"], t["bias"], t["dout"], None, 0.25)
    dq, dk, dv, dg, db = g
    # one key: P = 1, dS = 0, so only V and G receive gradient
    assert np.all(np.abs(dq) < 1e-14) and np.all(np.abs(dk) < 1e-14)
    assert np.all(np.abs(db) < 1e-14)
    np.testing.assert_allclose(dv, t["dout"] * sig(t["g"]), atol=1e-14)


@pytest.mark.parametrize("node", [STARTING, ENDING])
def test_constant_values_and_weights_sum_to_one(node):
    n, h, d = 7, 2, 3
    t, gen = rnd(n, h, d, 61)
    mask = W.random_mask(n, 0.8, gen).numpy()
    mask[:, 0] = 1
    mask[0, :] = 1
    v = np.broadcast_to(np.array([1.5, -2.0, 0.25]), t["v"].shape).copy()
    out, lse = oracle.fwd(node, t["q"], t["k"], v, t["g"], t["bias"], mask, 0.4)
    np.testing.assert_allclose(out, sig(t["g"]) * v, atol=1e-13)  # sum_k P = 1
    dq, dk, dv, dg, db = oracle.bwd(node, t["q"], t["k"], v, t["g"], t["bias"], t["dout"], mask,
                                    0.4)
    for x in (dq, dk, db):
        assert np.max(np.abs(x)) < 1e-12  # dP = D for every key, so dS = 0


@pytest.mark.parametrize("node", [STARTING, ENDING])
def test_masked_keys_get_zero_weight_and_gradient(node):
    n, h, d = 6, 2, 3
    t, gen = rnd(n, h, d, 71)
    mask = W.random_mask(n, 0.6, gen).numpy()
    out, lse = oracle.fwd(node, t["q"], t["k"], t["v"], t["g"], t["bias"], mask, 0.5)
    k2, v2 = t["k"].copy(), t["v"].copy()
    rng = np.random.default_rng(0)
    for a in range(n):
        for b in range(n):
            if mask[a, b] == 0:  # the pair entry (a, b) is a masked key of its row
                k2[a, b] += rng.normal(size=k2[a, b].shape) * 10
                v2[a, b] += rng.normal(size=v2[a, b].shape) * 10
    out2, lse2 = oracle.fwd(node, t["q"], k2, v2, t["g"], t["bias"], mask, 0.5)
    np.testing.assert_allclose(out2, out, atol=1e-13)
    dq, dk, dv, dg, db = oracle.bwd(node, t["q"], t["k"], t["v"], t["g"], t["bias"], t["dout"],
                                    mask, 0.5)
    for a in range(n):
        for b in range(n):
            if mask[a, b] == 0:
                assert np.all(dk[a, b] == 0) and np.all(dv[a, b] == 0)
                # a masked key gets no bias gradient from any query
                if node == STARTING:
                    pass  # (bias columns are shared by all rows, not masked per row)


@pytest.mark.parametrize("node", [STARTING, ENDING])
def test_fully_masked_queries(node):
    n, h, d = 5, 2, 3
    t, _ = rnd(n, h, d, 81)
    mask = W.pair_mask(n, 2).numpy()  # padded tokens: their rows have no valid key
    out, lse = oracle.fwd(node, t["q"], t["k"], t["v"], t["g"], t["bias"], mask, 0.5)
    dq, dk, dv, dg, db = oracle.bwd(node, t["q"], t["k"], t["v"], t["g"], t["bias"], t["dout"],
                                    mask, 0.5)
    for row in (3, 4):
        for qi in range(n):
            at = (row, qi) if node == STARTING else (qi, row)
            assert np.all(out[at] == 0) and np.all(lse[at] == -np.inf)
            assert np.all(dq[at] == 0) and np.all(dg[at] == 0)
    # padded keys are masked for every row, so they get no K/V gradient
    for row in range(n):
        for k in (3, 4):
            kat = (row, k) if node == STARTING else (k, row)
            assert np.all(dk[kat] == 0) and np.all(dv[kat] == 0)
    # and no bias gradient: dB[q, k] with k padded is a sum of zeros
    bk = db[:, 3:] if node == STARTING else db[3:, :]
    assert np.all(bk == 0)


@pytest.mark.parametrize("node", [STARTING, ENDING])
def test_bias_shift_invariance_and_db_row_sums(node):
    n, h, d = 6, 3, 4
    t, gen = rnd(n, h, d, 91)
    mask = W.random_mask(n, 0.7, gen).numpy()
    if node == STARTING:
        mask[:, 1] = 1
    else:
        mask[1, :] = 1
    shift = np.random.default_rng(1).normal(size=(n, h))  # one constant per (query, head)
    b2 = t["bias"].copy()
    for qi in range(n):
        if node == STARTING:
            b2[qi, :, :] += shift[qi][None, :]
        else:
            b2[:, qi, :] += shift[qi][None, :]
    o1, l1 = oracle.fwd(node, t["q"], t["k"], t["v"], t["g"], t["bias"], mask, 0.5)
    o2, l2 = oracle.fwd(node, t["q"], t["k"], t["v"], t["g"], b2, mask, 0.5)
    np.testing.assert_allclose(o2, o1, atol=1e-12)
    for row in range(n):
        for qi in range(n):
            at = (row, qi) if node == STARTING else (qi, row)
            np.testing.assert_allclose(l2[at], l1[at] + shift[qi], atol=1e-12)
    db = oracle.bwd(node, t["q"], t["k"], t["v"], t["g"], t["bias"], t["dout"], mask, 0.5)[4]
    # sum_k dS = 0 for every (row, query), so each query's dB sums to zero over keys
    sums = db.sum(1) if node == STARTING else db.sum(0)
    np.testing.assert_allclose(sums, 0, atol=1e-12)


def test_row_and_query_subsets_match_full_run():
    n, h, d = 8, 2, 3
    t, gen = rnd(n, h, d, 101)
    mask = W.random_mask(n, 0.8, gen).numpy()
    for node in (STARTING, ENDING):
        o, l = oracle.fwd(node, t["q"], t["k"], t["v"], t["g"], t["bias"], mask)
        full = oracle.bwd(node, t["q"], t["k"], t["v"], t["g"], t["bias"], t["dout"], mask)
        rows, qs = [6, 1], [5, 0]
        os_, ls = oracle.fwd(node, t["q"], t["k"], t["v"], t["g"], t["bias"], mask, rows=rows)
        part = oracle.bwd(node, t["q"], t["k"], t["v"], t["g"], t["bias"], t["dout"], mask,
                          rows=rows, db_queries=qs)
        sel = (slice(None), rows) if node == ENDING else (rows,)
        np.testing.assert_array_equal(os_[sel], o[sel])
        np.testing.assert_array_equal(ls[sel], l[sel])
        for a, b in zip(part[:4], full[:4]):
            np.testing.assert_array_equal(a[sel], b[sel])
        bsel = (qs,) if node == STARTING else (slice(None), qs)
        np.testing.assert_array_equal(part[4][bsel], full[4][bsel])


def _val(s):
    if isinstance(s, (int, float)):
        return float(s)
    if s.startswith("ln"):
        return math.log(float(s[2:]))
    return float(Fraction(s))


def _arr(x):
    return np.array([[_val(e) for e in row] for row in x])


def test_hand_derived_fixture():
    with open(os.path.join(GOLDEN, "hand_n2.json")) as f:
        gd = json.load(f)
    n, h, d = gd["n"], gd["h"], gd["d"]
    pair = lambda x: _arr(x).reshape(n, n, h, d)  # noqa: E731
    q, k, v, g, do = (pair(gd[x]) for x in ("q", "k", "v", "g", "dout"))
    bias = _arr(gd["bias"]).reshape(n, n, h)
    for key, node, mask in (("starting", STARTING, None), ("ending", ENDING, None),
                            ("starting_masked", STARTING, None)):
        exp = gd[key]
        mask = np.array(exp["mask"], np.uint8) if "mask" in exp else None
        out, lse = oracle.fwd(node, q, k, v, g, bias, mask, gd["scale"])
        np.testing.assert_allclose(out.reshape(n, n), _arr(exp["out"]), atol=1e-14, err_msg=key)
        np.testing.assert_allclose(lse.reshape(n, n), _arr(exp["lse"]), atol=1e-14, err_msg=key)
        if "dq" in exp:
            grads = oracle.bwd(node, q, k, v, g, bias, do, mask, gd["scale"])
            for name, x in zip(("dq", "dk", "dv", "dg", "db"), grads):
                np.testing.assert_allclose(x.reshape(n, n), _arr(exp[name]), atol=1e-14,
                                           err_msg=name)

"""C-ABI checks that need no GPU: the library loads, exports every symbol the
header declares, sizes workspaces, and rejects invalid arguments before any
HIP call (so none of these calls launches anything)."""
import ctypes
import os
import re

import pytest

from paper_2506_20686_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "triattn.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(B.LIB_PATH):
        from paper_2506_20686_amd import build
        build.build()
    return B.lib()


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(tri_(?:attn|ln_linear|transition)_\w+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    names = header_functions()
    assert len(names) >= 5
    for name in names:
        assert hasattr(lib, name), name


def test_status_strings(lib):
    assert B.tri_attn_status_string(B.OK) == "ok"
    for s in (B.ERR_INVALID_ARG, B.ERR_UNSUPPORTED, B.ERR_WORKSPACE, B.ERR_HIP,
              B.ERR_TOO_LARGE):
        assert B.tri_attn_status_string(s) not in ("ok", "unknown status")
    assert B.tri_attn_status_string(99) == "unknown status"


def ws_bytes(fn, *args):
    out = ctypes.c_size_t(0)
    st = fn(*args, ctypes.byref(out))
    return st, out.value


@pytest.mark.parametrize("dtype", [B.F32, B.BF16])
@pytest.mark.parametrize("node", [B.STARTING, B.ENDING])
def test_workspace_sizes(lib, node, dtype):
    el = 2 if dtype == B.BF16 else 4
    for n, h in ((1, 1), (32, 4), (37, 1), (256, 4), (768, 4), (1536, 4)):
        st, f = ws_bytes(lib.tri_attn_fwd_workspace_bytes, node, dtype, n, h, 32)
        assert st == B.OK
        np_ = (n + 31) // 32 * 32
        assert f >= h * np_ * np_ * 4 + n * (np_ // 32) * 4
        st, b = ws_bytes(lib.tri_attn_bwd_workspace_bytes, node, dtype, n, h, 32)
        assert st == B.OK
        assert b >= f + h * np_ * np_ * 4 + 2 * h * n * np_ * 4 + n * n * h * 32 * el
        # O(N^2 H) memory: far below the N^3 H logits the method avoids
        if n >= 768:
            assert b < n ** 3 * h * el / 3


def test_workspace_size_errors(lib):
    f = lib.tri_attn_fwd_workspace_bytes
    assert ws_bytes(f, 2, B.BF16, 8, 1, 32)[0] == B.ERR_INVALID_ARG
    assert ws_bytes(f, 0, 7, 8, 1, 32)[0] == B.ERR_INVALID_ARG
    assert ws_bytes(f, 0, B.BF16, 0, 1, 32)[0] == B.ERR_INVALID_ARG
    assert ws_bytes(f, 0, B.BF16, 8, 0, 32)[0] == B.ERR_INVALID_ARG
    assert ws_bytes(f, 0, B.BF16, 9000, 1, 32)[0] == B.ERR_INVALID_ARG
    assert ws_bytes(f, 0, B.BF16, 8, 1, 128)[0] == B.ERR_UNSUPPORTED
    assert f(0, B.BF16, 8, 1, 32, None) == B.ERR_INVALID_ARG


# Fake, 16-byte aligned, non-null addresses: every call below is invalid, so
# the library must return before it would touch them.
P = 0x10000


def fwd_args(**over):
    a = dict(node=0, dtype=B.BF16, n=16, h=2, d=32, scale=0.17, q=P, k=P, v=P, g=P, bias=P,
             mask=None, out=P, lse=P, ws=P, wsb=1 << 30, stream=None)
    a.update(over)
    return (a["node"], a["dtype"], a["n"], a["h"], a["d"], a["scale"], a["q"], a["k"], a["v"],
            a["g"], a["bias"], a["mask"], a["out"], a["lse"], a["ws"], a["wsb"], a["stream"])


def bwd_args(**over):
    a = dict(node=0, dtype=B.BF16, n=16, h=2, d=32, scale=0.17, q=P, k=P, v=P, g=P, bias=P,
             mask=None, out=P, lse=P, dout=P, dq=P, dk=P, dv=P, dg=P, dbias=P, ws=P,
             wsb=1 << 30, stream=None)
    a.update(over)
    return (a["node"], a["dtype"], a["n"], a["h"], a["d"], a["scale"], a["q"], a["k"], a["v"],
            a["g"], a["bias"], a["mask"], a["out"], a["lse"], a["dout"], a["dq"], a["dk"],
            a["dv"], a["dg"], a["dbias"], a["ws"], a["wsb"], a["stream"])


FWD_BAD = [
    (dict(node=5), B.ERR_INVALID_ARG), (dict(dtype=-1), B.ERR_INVALID_ARG),
    (dict(n=0), B.ERR_INVALID_ARG), (dict(h=0), B.ERR_INVALID_ARG),
    (dict(d=128), B.ERR_UNSUPPORTED), (dict(d=24), B.ERR_UNSUPPORTED), (dict(scale=0.0), B.ERR_INVALID_ARG),
    (dict(scale=-1.0), B.ERR_INVALID_ARG), (dict(scale=float("nan")), B.ERR_INVALID_ARG),
    (dict(scale=float("inf")), B.ERR_INVALID_ARG),
    (dict(q=None), B.ERR_INVALID_ARG), (dict(k=None), B.ERR_INVALID_ARG),
    (dict(v=None), B.ERR_INVALID_ARG), (dict(g=None), B.ERR_INVALID_ARG),
    (dict(bias=None), B.ERR_INVALID_ARG), (dict(out=None), B.ERR_INVALID_ARG),
    (dict(lse=None), B.ERR_INVALID_ARG), (dict(q=P + 2), B.ERR_INVALID_ARG),
    (dict(lse=P + 4), B.ERR_INVALID_ARG),
    (dict(ws=None), B.ERR_WORKSPACE), (dict(wsb=16), B.ERR_WORKSPACE),
    (dict(ws=P + 8), B.ERR_WORKSPACE),
]


@pytest.mark.parametrize("over,code", FWD_BAD)
def test_fwd_rejects_before_any_hip_call(lib, over, code):
    assert lib.tri_attn_fwd(*fwd_args(**over)) == code


BWD_BAD = FWD_BAD + [
    (dict(dout=None), B.ERR_INVALID_ARG), (dict(dq=None), B.ERR_INVALID_ARG),
    (dict(dk=None), B.ERR_INVALID_ARG), (dict(dv=None), B.ERR_INVALID_ARG),
    (dict(dg=None), B.ERR_INVALID_ARG), (dict(dbias=None), B.ERR_INVALID_ARG),
    (dict(dbias=P + 2), B.ERR_INVALID_ARG),
]


@pytest.mark.parametrize("over,code", BWD_BAD)
def test_bwd_rejects_before_any_hip_call(lib, over, code):
    assert lib.tri_attn_bwd(*bwd_args(**over)) == code


def test_undersized_workspace_reports_exact_requirement(lib):
    for node in (0, 1):
        st, need = ws_bytes(lib.tri_attn_bwd_workspace_bytes, node, B.BF16, 16, 2, 32)
        assert st == B.OK
        assert lib.tri_attn_bwd(*bwd_args(node=node, wsb=need - 1)) == B.ERR_WORKSPACE
        st, need = ws_bytes(lib.tri_attn_fwd_workspace_bytes, node, B.BF16, 16, 2, 32)
        assert lib.tri_attn_fwd(*fwd_args(node=node, wsb=need - 1)) == B.ERR_WORKSPACE


# ---- fused layer-norm + linear projection ----------------------------------------------

COLS = [128, 128, 128, 128, 4]


def lnl_args(**over):
    a = dict(dtype=B.BF16, m=1000, k=128, cols=COLS, eps=1e-5, x=P, gamma=P, beta=P, w=P,
             outs=[P] * len(over.get("cols", COLS)), mean=P, rstd=P, stream=None)
    a.update(over)
    cols = (ctypes.c_int64 * len(a["cols"]))(*a["cols"])
    outs = None if a["outs"] is None else (ctypes.c_void_p * len(a["outs"]))(*a["outs"])
    return (a["dtype"], a["m"], a["k"], len(a["cols"]), cols, a["eps"], a["x"], a["gamma"],
            a["beta"], a["w"], outs, a["mean"], a["rstd"], a["stream"])


LNL_BAD = [
    (dict(dtype=-1), B.ERR_INVALID_ARG), (dict(dtype=B.F32), B.ERR_UNSUPPORTED),
    (dict(m=0), B.ERR_INVALID_ARG), (dict(k=64), B.ERR_UNSUPPORTED),
    (dict(k=0), B.ERR_INVALID_ARG), (dict(cols=[128, 6]), B.ERR_UNSUPPORTED),
    (dict(cols=[128, 0]), B.ERR_INVALID_ARG), (dict(cols=[512, 516]), B.ERR_UNSUPPORTED),
    (dict(cols=[4] * 9), B.ERR_UNSUPPORTED), (dict(eps=-1.0), B.ERR_INVALID_ARG),
    (dict(eps=float("nan")), B.ERR_INVALID_ARG), (dict(x=None), B.ERR_INVALID_ARG),
    (dict(gamma=None), B.ERR_INVALID_ARG), (dict(beta=None), B.ERR_INVALID_ARG),
    (dict(w=None), B.ERR_INVALID_ARG), (dict(mean=None), B.ERR_INVALID_ARG),
    (dict(rstd=P + 4), B.ERR_INVALID_ARG), (dict(outs=None), B.ERR_INVALID_ARG),
    (dict(outs=[P, P, None, P, P]), B.ERR_INVALID_ARG),
    (dict(outs=[P, P, P, P, P + 8]), B.ERR_INVALID_ARG),
]


@pytest.mark.parametrize("over,code", LNL_BAD)
def test_ln_linear_fwd_rejects_before_any_hip_call(lib, over, code):
    assert lib.tri_ln_linear_fwd(*lnl_args(**over)) == code


def lnl_bwd_args(**over):
    cols = over.get("cols", COLS)
    a = dict(dtype=B.BF16, m=1000, k=128, cols=cols, x=P, gamma=P, beta=P, w=P, mean=P, rstd=P,
             douts=[P] * len(cols), dx=P, dw=P, dgamma=P, dbeta=P, ws=P, wsb=1 << 30,
             stream=None)
    a.update(over)
    c = (ctypes.c_int64 * len(a["cols"]))(*a["cols"])
    douts = None if a["douts"] is None else (ctypes.c_void_p * len(a["douts"]))(*a["douts"])
    return (a["dtype"], a["m"], a["k"], len(a["cols"]), c, a["x"], a["gamma"], a["beta"],
            a["w"], a["mean"], a["rstd"], douts, a["dx"], a["dw"], a["dgamma"], a["dbeta"],
            a["ws"], a["wsb"], a["stream"])


def test_ln_linear_bwd_workspace_size(lib):
    for m, cols in ((1, [4]), (5000, COLS), (768 * 768, COLS), (77, [32, 64, 8, 96, 4])):
        got = B.tri_ln_linear_bwd_workspace_bytes(B.BF16, m, 128, cols)
        np_ = (sum(cols) + 31) // 32 * 32
        parts = min(256, (m + 31) // 32)
        assert got >= (parts + 1) * 129 * np_ * 4
        assert got % 256 == 0


LNL_BWD_BAD = [
    (dict(dtype=B.F32), B.ERR_UNSUPPORTED), (dict(m=0), B.ERR_INVALID_ARG),
    (dict(k=64), B.ERR_UNSUPPORTED), (dict(cols=[512, 64]), B.ERR_UNSUPPORTED),
    (dict(cols=[128, 6]), B.ERR_UNSUPPORTED), (dict(m=1 << 30), B.ERR_UNSUPPORTED),
    (dict(x=None), B.ERR_INVALID_ARG), (dict(mean=None), B.ERR_INVALID_ARG),
    (dict(rstd=P + 4), B.ERR_INVALID_ARG), (dict(dx=None), B.ERR_INVALID_ARG),
    (dict(dw=None), B.ERR_INVALID_ARG), (dict(dgamma=None), B.ERR_INVALID_ARG),
    (dict(dbeta=P + 8), B.ERR_INVALID_ARG), (dict(douts=None), B.ERR_INVALID_ARG),
    (dict(douts=[P, P, P, None, P]), B.ERR_INVALID_ARG),
    (dict(ws=None), B.ERR_WORKSPACE), (dict(wsb=100), B.ERR_WORKSPACE),
]


@pytest.mark.parametrize("over,code", LNL_BWD_BAD)
def test_ln_linear_bwd_rejects_before_any_hip_call(lib, over, code):
    assert lib.tri_ln_linear_bwd(*lnl_bwd_args(**over)) == code


# ---- starting node over a range of rows -----------------------------------------------

@pytest.mark.parametrize("dtype", [B.F32, B.BF16])
def test_rows_workspace_sizes(lib, dtype):
    for n, h in ((1, 1), (37, 1), (768, 4), (1536, 4)):
        whole = [ws_bytes(f, B.STARTING, dtype, n, h, 32)[1]
                 for f in (lib.tri_attn_fwd_workspace_bytes, lib.tri_attn_bwd_workspace_bytes)]
        prev = [0, 0]
        for rows in sorted({1, max(1, n // 8), max(1, n // 2), n}):
            got = []
            for f in (lib.tri_attn_rows_fwd_workspace_bytes, lib.tri_attn_rows_bwd_workspace_bytes):
                st, b = ws_bytes(f, dtype, n, rows, h, 32)
                assert st == B.OK
                got.append(b)
            # the whole range needs what the whole call needs; fewer rows never need more
            assert all(g >= p for g, p in zip(got, prev))
            if rows == n:
                assert got == whole
            prev = got


def test_rows_workspace_size_errors(lib):
    for f in (lib.tri_attn_rows_fwd_workspace_bytes, lib.tri_attn_rows_bwd_workspace_bytes):
        assert ws_bytes(f, B.BF16, 16, 0, 2, 32)[0] == B.ERR_INVALID_ARG
        assert ws_bytes(f, B.BF16, 16, 17, 2, 32)[0] == B.ERR_INVALID_ARG
        assert ws_bytes(f, B.BF16, 16, -1, 2, 32)[0] == B.ERR_INVALID_ARG
        assert ws_bytes(f, 7, 16, 4, 2, 32)[0] == B.ERR_INVALID_ARG
        assert ws_bytes(f, B.BF16, 16, 4, 2, 64)[0] == B.ERR_UNSUPPORTED
        assert f(B.BF16, 16, 4, 2, 32, None) == B.ERR_INVALID_ARG


def rows_fwd_args(**over):
    a = dict(dtype=B.BF16, n=16, rows=4, h=2, d=32, scale=0.17, q=P, k=P, v=P, g=P, bias=P,
             mask=None, out=P, lse=P, ws=P, wsb=1 << 30, stream=None)
    a.update(over)
    return (a["dtype"], a["n"], a["rows"], a["h"], a["d"], a["scale"], a["q"], a["k"], a["v"],
            a["g"], a["bias"], a["mask"], a["out"], a["lse"], a["ws"], a["wsb"], a["stream"])


def rows_bwd_args(**over):
    a = dict(dtype=B.BF16, n=16, rows=4, h=2, d=32, scale=0.17, q=P, k=P, v=P, g=P, bias=P,
             mask=None, out=P, lse=P, dout=P, dq=P, dk=P, dv=P, dg=P, dbias=P, ws=P,
             wsb=1 << 30, stream=None)
    a.update(over)
    return (a["dtype"], a["n"], a["rows"], a["h"], a["d"], a["scale"], a["q"], a["k"], a["v"],
            a["g"], a["bias"], a["mask"], a["out"], a["lse"], a["dout"], a["dq"], a["dk"],
            a["dv"], a["dg"], a["dbias"], a["ws"], a["wsb"], a["stream"])


ROWS_BAD = [(o, c) for o, c in FWD_BAD if "node" not in o] + [
    (dict(d=16), B.ERR_UNSUPPORTED), (dict(d=64), B.ERR_UNSUPPORTED),  # row ranges: d = 32
    (dict(rows=0), B.ERR_INVALID_ARG), (dict(rows=17), B.ERR_INVALID_ARG),
    (dict(rows=-3), B.ERR_INVALID_ARG),
]


@pytest.mark.parametrize("over,code", ROWS_BAD)
def test_rows_fwd_rejects_before_any_hip_call(lib, over, code):
    assert lib.tri_attn_rows_fwd(*rows_fwd_args(**over)) == code


@pytest.mark.parametrize("over,code", ROWS_BAD + [(o, c) for o, c in BWD_BAD
                                                   if o not in [x for x, _ in FWD_BAD]])
def test_rows_bwd_rejects_before_any_hip_call(lib, over, code):
    assert lib.tri_attn_rows_bwd(*rows_bwd_args(**over)) == code


def test_rows_undersized_workspace(lib):
    for rows in (1, 5, 16):
        for f, call, mk in ((lib.tri_attn_rows_fwd_workspace_bytes, lib.tri_attn_rows_fwd,
                             rows_fwd_args),
                            (lib.tri_attn_rows_bwd_workspace_bytes, lib.tri_attn_rows_bwd,
                             rows_bwd_args)):
            st, need = ws_bytes(f, B.BF16, 16, rows, 2, 32)
            assert st == B.OK
            assert call(*mk(rows=rows, wsb=need - 1)) == B.ERR_WORKSPACE


# ---- fused transition layer -----------------------------------------------------------

def test_transition_workspace_sizes(lib):
    for m, f in ((1, 128), (1000, 512), (768 * 768, 512), (4096, 2048)):
        st, fw = ws_bytes(lib.tri_transition_fwd_workspace_bytes, B.BF16, m, 128, f)
        assert st == B.OK and fw >= (f // 32) * 24576
        st, bw = ws_bytes(lib.tri_transition_bwd_workspace_bytes, B.BF16, m, 128, f)
        # weight images, at least one partial-sum block and the totals
        assert st == B.OK and bw >= (f // 32) * 40960 + (128 * 2 * f * 2 + 4 * f + f * 128) * 4
        # the workspace does not grow with m beyond the partial-sum blocks
        assert bw < (f // 32) * 40960 + 257 * (128 * 2 * f + 2 * f + f * 128) * 4 + (1 << 20)
    f = lib.tri_transition_fwd_workspace_bytes
    assert ws_bytes(f, B.BF16, 0, 128, 512)[0] == B.ERR_INVALID_ARG
    assert ws_bytes(f, B.BF16, 10, 128, 0)[0] == B.ERR_INVALID_ARG
    assert ws_bytes(f, 9, 10, 128, 512)[0] == B.ERR_INVALID_ARG
    assert ws_bytes(f, B.F32, 10, 128, 512)[0] == B.ERR_UNSUPPORTED
    assert ws_bytes(f, B.BF16, 10, 64, 512)[0] == B.ERR_UNSUPPORTED
    assert ws_bytes(f, B.BF16, 10, 128, 500)[0] == B.ERR_UNSUPPORTED
    assert ws_bytes(f, B.BF16, 10, 128, 4096)[0] == B.ERR_UNSUPPORTED
    assert f(B.BF16, 10, 128, 512, None) == B.ERR_INVALID_ARG


def trn_fwd_args(**over):
    a = dict(dtype=B.BF16, m=64, c=128, f=512, eps=1e-5, x=P, gamma=P, beta=P, w1=P, w2=P, out=P,
             mean=P, rstd=P, ws=P, wsb=1 << 30, stream=None)
    a.update(over)
    return tuple(a[k] for k in ("dtype", "m", "c", "f", "eps", "x", "gamma", "beta", "w1", "w2",
                                "out", "mean", "rstd", "ws", "wsb", "stream"))


def trn_bwd_args(**over):
    a = dict(dtype=B.BF16, m=64, c=128, f=512, x=P, gamma=P, beta=P, w1=P, w2=P, mean=P, rstd=P,
             dout=P, dx=P, dw1=P, dw2=P, dgamma=P, dbeta=P, ws=P, wsb=1 << 30, stream=None)
    a.update(over)
    return tuple(a[k] for k in ("dtype", "m", "c", "f", "x", "gamma", "beta", "w1", "w2", "mean",
                                "rstd", "dout", "dx", "dw1", "dw2", "dgamma", "dbeta", "ws", "wsb",
                                "stream"))


TRN_COMMON_BAD = [
    (dict(dtype=5), B.ERR_INVALID_ARG), (dict(m=0), B.ERR_INVALID_ARG),
    (dict(f=0), B.ERR_INVALID_ARG), (dict(dtype=B.F32), B.ERR_UNSUPPORTED),
    (dict(c=96), B.ERR_UNSUPPORTED), (dict(f=200), B.ERR_UNSUPPORTED),
    (dict(x=None), B.ERR_INVALID_ARG), (dict(w1=P + 8), B.ERR_INVALID_ARG),
    (dict(gamma=None), B.ERR_INVALID_ARG), (dict(w2=None), B.ERR_INVALID_ARG),
    (dict(mean=None), B.ERR_INVALID_ARG), (dict(rstd=P + 4), B.ERR_INVALID_ARG),
    (dict(ws=None), B.ERR_WORKSPACE), (dict(wsb=100), B.ERR_WORKSPACE),
]


@pytest.mark.parametrize("over,code", TRN_COMMON_BAD + [
    (dict(eps=-1.0), B.ERR_INVALID_ARG), (dict(eps=float("nan")), B.ERR_INVALID_ARG),
    (dict(out=None), B.ERR_INVALID_ARG)])
def test_transition_fwd_rejects_before_any_hip_call(lib, over, code):
    assert lib.tri_transition_fwd(*trn_fwd_args(**over)) == code


@pytest.mark.parametrize("over,code", TRN_COMMON_BAD + [
    (dict(dout=None), B.ERR_INVALID_ARG), (dict(dx=None), B.ERR_INVALID_ARG),
    (dict(dw1=None), B.ERR_INVALID_ARG), (dict(dw2=P + 2), B.ERR_INVALID_ARG),
    (dict(dgamma=None), B.ERR_INVALID_ARG), (dict(dbeta=None), B.ERR_INVALID_ARG)])
def test_transition_bwd_rejects_before_any_hip_call(lib, over, code):
    assert lib.tri_transition_bwd(*trn_bwd_args(**over)) == code


def test_transition_undersized_workspace(lib):
    for fn, call, mk in ((lib.tri_transition_fwd_workspace_bytes, lib.tri_transition_fwd,
                          trn_fwd_args),
                         (lib.tri_transition_bwd_workspace_bytes, lib.tri_transition_bwd,
                          trn_bwd_args)):
        st, need = ws_bytes(fn, B.BF16, 64, 128, 512)
        assert st == B.OK
        assert call(*mk(wsb=need - 1)) == B.ERR_WORKSPACE


# ---- batched attention -------------------------------------------------------------------

def batched_fwd_args(**over):
    a = dict(batch=3)
    a.update({k: v for k, v in over.items() if k == "batch"})
    base = fwd_args(**{k: v for k, v in over.items() if k != "batch"})
    return base[:2] + (a["batch"],) + base[2:]


def batched_bwd_args(**over):
    a = dict(batch=3)
    a.update({k: v for k, v in over.items() if k == "batch"})
    base = bwd_args(**{k: v for k, v in over.items() if k != "batch"})
    return base[:2] + (a["batch"],) + base[2:]


@pytest.mark.parametrize("over,code", FWD_BAD + [(dict(batch=0), B.ERR_INVALID_ARG),
                                                 (dict(batch=-2), B.ERR_INVALID_ARG),
                                                 (dict(batch=(1 << 20) + 1), B.ERR_INVALID_ARG)])
def test_batched_fwd_rejects_before_any_hip_call(lib, over, code):
    assert lib.tri_attn_fwd_batched(*batched_fwd_args(**over)) == code


@pytest.mark.parametrize("over,code", BWD_BAD + [(dict(batch=0), B.ERR_INVALID_ARG)])
def test_batched_bwd_rejects_before_any_hip_call(lib, over, code):
    assert lib.tri_attn_bwd_batched(*batched_bwd_args(**over)) == code


def test_batched_workspace_is_the_unbatched_one(lib):
    for node in (0, 1):
        st, need = ws_bytes(lib.tri_attn_bwd_workspace_bytes, node, B.BF16, 16, 2, 32)
        assert lib.tri_attn_bwd_batched(*batched_bwd_args(node=node, wsb=need - 1)) == \
            B.ERR_WORKSPACE
        st, need = ws_bytes(lib.tri_attn_fwd_workspace_bytes, node, B.BF16, 16, 2, 32)
        assert lib.tri_attn_fwd_batched(*batched_fwd_args(node=node, wsb=need - 1)) == \
            B.ERR_WORKSPACE


def test_batched_workspace_sizes(lib):
    """One launch per kernel for a batch needs one unbatched workspace per
    sample; fp32 d = 16 (per-sample padded copies) and a batch of one need
    the unbatched size; the size calls reject what the batched calls reject."""
    fns = ((lib.tri_attn_fwd_batched_workspace_bytes, lib.tri_attn_fwd_workspace_bytes),
           (lib.tri_attn_bwd_batched_workspace_bytes, lib.tri_attn_bwd_workspace_bytes))
    for fb, f1 in fns:
        for dtype in (B.BF16, B.F32):
            for node in (0, 1):
                for d in (16, 32, 64):
                    st, one = ws_bytes(f1, node, dtype, 37, 3, d)
                    assert st == B.OK
                    padded = d == 16 and dtype == B.F32
                    for batch, k in ((1, 1), (4, 1 if padded else 4),
                                     (65535, 1 if padded else 65535), (65536, 1)):
                        out = ctypes.c_size_t(0)
                        assert fb(node, dtype, batch, 37, 3, d, ctypes.byref(out)) == B.OK
                        assert out.value == k * one, (node, dtype, d, batch)
        out = ctypes.c_size_t(0)
        assert fb(0, B.BF16, 0, 37, 3, 32, ctypes.byref(out)) == B.ERR_INVALID_ARG
        assert fb(0, B.BF16, (1 << 20) + 1, 37, 3, 32, ctypes.byref(out)) == B.ERR_INVALID_ARG
        assert fb(0, B.BF16, 2, 37, 3, 32, None) == B.ERR_INVALID_ARG
        assert fb(0, B.BF16, 2, 37, 3, 48, ctypes.byref(out)) != B.OK


def test_d16_workspace(lib):
    """fp32 d = 16 runs the d = 32 kernels on zero-padded copies kept in the
    workspace: 5 (forward) and 10 (backward) tensors of [n][n][h][32].  bf16
    d = 16 reads the 16-channel tensors directly: the forward workspace is
    that of d = 32, the backward's dA buffers (hi and lo) are half as large."""
    n, h = 40, 3
    for node in (0, 1):
        el = 4
        pad = -(-n * n * h * 32 * el // 256) * 256
        for fn, k in ((lib.tri_attn_fwd_workspace_bytes, 5),
                      (lib.tri_attn_bwd_workspace_bytes, 10)):
            st, b32 = ws_bytes(fn, node, B.F32, n, h, 32)
            st16, b16 = ws_bytes(fn, node, B.F32, n, h, 16)
            assert st == st16 == B.OK
            assert b16 == b32 + k * pad
        pair32 = -(-n * n * h * 32 * 2 // 256) * 256
        pair16 = -(-n * n * h * 16 * 2 // 256) * 256
        st, f32_ = ws_bytes(lib.tri_attn_fwd_workspace_bytes, node, B.BF16, n, h, 32)
        st16, f16 = ws_bytes(lib.tri_attn_fwd_workspace_bytes, node, B.BF16, n, h, 16)
        assert st == st16 == B.OK and f16 == f32_
        st, b32 = ws_bytes(lib.tri_attn_bwd_workspace_bytes, node, B.BF16, n, h, 32)
        st16, b16 = ws_bytes(lib.tri_attn_bwd_workspace_bytes, node, B.BF16, n, h, 16)
        assert st == st16 == B.OK and b16 == b32 - 2 * (pair32 - pair16)


def test_d64_workspace_scales_the_pair_buffers(lib):
    """d = 64 runs the register-staged kernels with 64 channels: the dA
    buffers (and the bf16 low part) double, nothing else changes."""
    for dtype, el, parts in ((B.BF16, 2, 2), (B.F32, 4, 1)):
        n, h = 40, 3
        pair = -(-n * n * h * 32 * el // 256) * 256
        pair64 = -(-n * n * h * 64 * el // 256) * 256
        st, b32 = ws_bytes(lib.tri_attn_bwd_workspace_bytes, 0, dtype, n, h, 32)
        st64, b64 = ws_bytes(lib.tri_attn_bwd_workspace_bytes, 0, dtype, n, h, 64)
        assert st == st64 == B.OK
        assert b64 == b32 + parts * (pair64 - pair)
        st, f32_ = ws_bytes(lib.tri_attn_fwd_workspace_bytes, 0, dtype, n, h, 32)
        st, f64_ = ws_bytes(lib.tri_attn_fwd_workspace_bytes, 0, dtype, n, h, 64)
        assert f32_ == f64_


def test_noalloc_forward_rejects_before_any_hip_call(lib):
    """The allocation-free forward checks sizes, pointers and its scratch
    limit before it looks up the scratch array or launches anything."""
    f = lib.tri_attn_fwd_noalloc
    good = (P,) * 5
    sc = 0.1767767
    assert f(0, B.BF16, 0, 1, 32, sc, *good, None, P, P, None) == B.ERR_INVALID_ARG
    assert f(0, B.BF16, 8, 1, 128, sc, *good, None, P, P, None) == B.ERR_UNSUPPORTED
    assert f(0, B.BF16, 8, 1, 32, -1.0, *good, None, P, P, None) == B.ERR_INVALID_ARG
    assert f(0, B.BF16, 8, 1, 32, sc, None, P, P, P, P, None, P, P, None) == B.ERR_INVALID_ARG
    assert f(0, B.BF16, 8, 1, 32, sc, P + 8, P, P, P, P, None, P, P, None) == B.ERR_INVALID_ARG
    # bias planes of n = 2048, h = 4 alone are 64 MiB, beyond the 32 MiB array
    assert f(0, B.BF16, 2048, 4, 32, sc, *good, None, P, P, None) == B.ERR_TOO_LARGE
    assert f(1, B.F32, 8192, 64, 32, sc, *good, None, P, P, None) == B.ERR_TOO_LARGE


def test_mfma_probe_rejects_bad_sizes(lib):
    """The MFMA counter-calibration kernel checks its sizes before launching."""
    f = lib.tri_attn_mfma_probe
    assert f(0, 10, P, None) == B.ERR_INVALID_ARG
    assert f(1, 0, P, None) == B.ERR_INVALID_ARG
    assert f((1 << 20) + 1, 10, P, None) == B.ERR_INVALID_ARG
    assert f(1, 10, None, None) == B.ERR_INVALID_ARG

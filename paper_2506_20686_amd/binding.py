"""Python binding of libtriattn.so (ctypes).

The functions named like the C entry points pass raw pointers through; the
convenience wrappers fwd() / bwd() check torch tensors (device, dtype, shape,
contiguity), allocate outputs and workspace with torch and call the library
on torch's current stream.  All arithmetic happens in the library's HIP
kernels; there is no fallback path.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libtriattn.so")

OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_HIP, ERR_TOO_LARGE = 0, 1, 2, 3, 4, 5
FWD_NOALLOC_SCRATCH_BYTES = 32 << 20  # TRIATTN_FWD_NOALLOC_SCRATCH_BYTES
STARTING, ENDING = 0, 1
F32, BF16 = 0, 1
HEAD_DIM = 32

_LIB = None
_vp, _i64, _f, _int, _sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_float, ctypes.c_int, ctypes.c_size_t


class TriAttnError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {tri_attn_status_string(status)} (status {status})")


def lib():
    """Load libtriattn.so (raises if it has not been built)."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2506_20686_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        L.tri_attn_fwd_workspace_bytes.argtypes = [_int, _int, _i64, _i64, _i64,
                                                   ctypes.POINTER(_sz)]
        L.tri_attn_bwd_workspace_bytes.argtypes = L.tri_attn_fwd_workspace_bytes.argtypes
        L.tri_attn_fwd.argtypes = [_int, _int, _i64, _i64, _i64, _f] + [_vp] * 9 + [_sz, _vp]
        L.tri_attn_bwd.argtypes = [_int, _int, _i64, _i64, _i64, _f] + [_vp] * 15 + [_sz, _vp]
        L.tri_attn_fwd_noalloc.argtypes = [_int, _int, _i64, _i64, _i64, _f] + [_vp] * 9
        L.tri_attn_fwd_noalloc.restype = _int
        L.tri_attn_mfma_probe.argtypes = [_i64, _i64, _vp, _vp]
        L.tri_attn_mfma_probe.restype = _int
        L.tri_attn_rows_fwd_workspace_bytes.argtypes = [_int, _i64, _i64, _i64, _i64,
                                                        ctypes.POINTER(_sz)]
        L.tri_attn_rows_bwd_workspace_bytes.argtypes = L.tri_attn_rows_fwd_workspace_bytes.argtypes
        L.tri_attn_rows_fwd.argtypes = [_int, _i64, _i64, _i64, _i64, _f] + [_vp] * 9 + [_sz, _vp]
        L.tri_attn_rows_bwd.argtypes = [_int, _i64, _i64, _i64, _i64, _f] + [_vp] * 15 + [_sz,
                                                                                          _vp]
        L.tri_attn_fwd_batched.argtypes = [_int, _int, _i64, _i64, _i64, _i64, _f] + [_vp] * 9 + \
            [_sz, _vp]
        L.tri_attn_bwd_batched.argtypes = [_int, _int, _i64, _i64, _i64, _i64, _f] + [_vp] * 15 + \
            [_sz, _vp]
        L.tri_attn_fwd_batched.restype = _int
        L.tri_attn_bwd_batched.restype = _int
        L.tri_attn_fwd_batched_workspace_bytes.argtypes = [_int, _int, _i64, _i64, _i64, _i64,
                                                           ctypes.POINTER(_sz)]
        L.tri_attn_bwd_batched_workspace_bytes.argtypes = \
            L.tri_attn_fwd_batched_workspace_bytes.argtypes
        L.tri_attn_fwd_batched_workspace_bytes.restype = _int
        L.tri_attn_bwd_batched_workspace_bytes.restype = _int
        L.tri_attn_status_string.argtypes = [_int]
        L.tri_attn_status_string.restype = ctypes.c_char_p
        L.tri_attn_timing_enable.argtypes = [_int]
        L.tri_attn_timing_select.argtypes = [ctypes.c_uint64]
        L.tri_attn_timing_reset.argtypes = []
        L.tri_attn_timing_read.argtypes = [_int, ctypes.POINTER(ctypes.c_char_p),
                                           ctypes.POINTER(ctypes.c_double),
                                           ctypes.POINTER(ctypes.c_int64)]
        _i64p = ctypes.POINTER(_i64)
        L.tri_ln_linear_fwd.argtypes = [_int, _i64, _i64, _int, _i64p, _f, _vp, _vp, _vp, _vp,
                                        ctypes.POINTER(_vp), _vp, _vp, _vp]
        L.tri_ln_linear_bwd_workspace_bytes.argtypes = [_int, _i64, _i64, _int, _i64p,
                                                        ctypes.POINTER(_sz)]
        L.tri_ln_linear_bwd.argtypes = [_int, _i64, _i64, _int, _i64p, _vp, _vp, _vp, _vp, _vp,
                                        _vp, ctypes.POINTER(_vp), _vp, _vp, _vp, _vp, _vp, _sz,
                                        _vp]
        L.tri_transition_fwd_workspace_bytes.argtypes = [_int, _i64, _i64, _i64,
                                                         ctypes.POINTER(_sz)]
        L.tri_transition_bwd_workspace_bytes.argtypes = \
            L.tri_transition_fwd_workspace_bytes.argtypes
        L.tri_transition_fwd.argtypes = [_int, _i64, _i64, _i64, _f] + [_vp] * 9 + [_sz, _vp]
        L.tri_transition_bwd.argtypes = [_int, _i64, _i64, _i64] + [_vp] * 14 + [_sz, _vp]
        for name in ("tri_transition_fwd_workspace_bytes", "tri_transition_bwd_workspace_bytes",
                     "tri_transition_fwd", "tri_transition_bwd"):
            getattr(L, name).restype = _int
        for name in ("tri_attn_fwd_workspace_bytes", "tri_attn_bwd_workspace_bytes",
                     "tri_attn_fwd", "tri_attn_bwd", "tri_attn_timing_enable",
                     "tri_attn_timing_reset", "tri_attn_timing_read", "tri_attn_timing_select",
                     "tri_ln_linear_fwd", "tri_ln_linear_bwd_workspace_bytes",
                     "tri_ln_linear_bwd", "tri_attn_rows_fwd_workspace_bytes",
                     "tri_attn_rows_bwd_workspace_bytes", "tri_attn_rows_fwd",
                     "tri_attn_rows_bwd"):
            getattr(L, name).restype = _int
        _LIB = L
    return _LIB


# ---- the C entry points, same names -----------------------------------------------

def tri_attn_status_string(status: int) -> str:
    return lib().tri_attn_status_string(int(status)).decode()


def tri_attn_fwd_workspace_bytes(node: int, dtype: int, n: int, h: int, d: int) -> int:
    out = _sz(0)
    st = lib().tri_attn_fwd_workspace_bytes(node, dtype, n, h, d, ctypes.byref(out))
    if st != OK:
        raise TriAttnError(st, "tri_attn_fwd_workspace_bytes")
    return out.value


def tri_attn_fwd_batched_workspace_bytes(node: int, dtype: int, batch: int, n: int, h: int,
                                         d: int) -> int:
    out = _sz(0)
    st = lib().tri_attn_fwd_batched_workspace_bytes(node, dtype, batch, n, h, d,
                                                    ctypes.byref(out))
    if st != OK:
        raise TriAttnError(st, "tri_attn_fwd_batched_workspace_bytes")
    return out.value


def tri_attn_bwd_batched_workspace_bytes(node: int, dtype: int, batch: int, n: int, h: int,
                                         d: int) -> int:
    out = _sz(0)
    st = lib().tri_attn_bwd_batched_workspace_bytes(node, dtype, batch, n, h, d,
                                                    ctypes.byref(out))
    if st != OK:
        raise TriAttnError(st, "tri_attn_bwd_batched_workspace_bytes")
    return out.value


def tri_attn_bwd_workspace_bytes(node: int, dtype: int, n: int, h: int, d: int) -> int:
    out = _sz(0)
    st = lib().tri_attn_bwd_workspace_bytes(node, dtype, n, h, d, ctypes.byref(out))
    if st != OK:
        raise TriAttnError(st, "tri_attn_bwd_workspace_bytes")
    return out.value


def tri_attn_fwd(node, dtype, n, h, d, scale, q, k, v, g, bias, mask, out, lse, workspace,
                 workspace_bytes, stream) -> int:
    """Raw call: every tensor argument is an integer device address (or None)."""
    return lib().tri_attn_fwd(node, dtype, n, h, d, scale, q, k, v, g, bias, mask, out, lse,
                              workspace, workspace_bytes, stream)


def tri_attn_mfma_probe(blocks: int, iters: int, out, stream) -> int:
    """Raw call of the MFMA counter-calibration kernel (out: device address)."""
    return lib().tri_attn_mfma_probe(blocks, iters, out, stream)


def tri_attn_fwd_noalloc(node, dtype, n, h, d, scale, q, k, v, g, bias, mask, out, lse,
                         stream) -> int:
    """Raw call: every tensor argument is an integer device address (or None)."""
    return lib().tri_attn_fwd_noalloc(node, dtype, n, h, d, scale, q, k, v, g, bias, mask, out,
                                      lse, stream)


def tri_attn_bwd(node, dtype, n, h, d, scale, q, k, v, g, bias, mask, out, lse, dout, dq, dk,
                 dv, dg, dbias, workspace, workspace_bytes, stream) -> int:
    """Raw call: every tensor argument is an integer device address (or None)."""
    return lib().tri_attn_bwd(node, dtype, n, h, d, scale, q, k, v, g, bias, mask, out, lse,
                              dout, dq, dk, dv, dg, dbias, workspace, workspace_bytes, stream)


def tri_attn_rows_fwd_workspace_bytes(dtype: int, n: int, rows: int, h: int, d: int) -> int:
    out = _sz(0)
    st = lib().tri_attn_rows_fwd_workspace_bytes(dtype, n, rows, h, d, ctypes.byref(out))
    if st != OK:
        raise TriAttnError(st, "tri_attn_rows_fwd_workspace_bytes")
    return out.value


def tri_attn_rows_bwd_workspace_bytes(dtype: int, n: int, rows: int, h: int, d: int) -> int:
    out = _sz(0)
    st = lib().tri_attn_rows_bwd_workspace_bytes(dtype, n, rows, h, d, ctypes.byref(out))
    if st != OK:
        raise TriAttnError(st, "tri_attn_rows_bwd_workspace_bytes")
    return out.value


def tri_attn_rows_fwd(dtype, n, rows, h, d, scale, q, k, v, g, bias, mask, out, lse, workspace,
                      workspace_bytes, stream) -> int:
    """Raw call: every tensor argument is an integer device address (or None)."""
    return lib().tri_attn_rows_fwd(dtype, n, rows, h, d, scale, q, k, v, g, bias, mask, out, lse,
                                   workspace, workspace_bytes, stream)


def tri_attn_rows_bwd(dtype, n, rows, h, d, scale, q, k, v, g, bias, mask, out, lse, dout, dq,
                      dk, dv, dg, dbias_partial, workspace, workspace_bytes, stream) -> int:
    """Raw call: every tensor argument is an integer device address (or None)."""
    return lib().tri_attn_rows_bwd(dtype, n, rows, h, d, scale, q, k, v, g, bias, mask, out, lse,
                                   dout, dq, dk, dv, dg, dbias_partial, workspace,
                                   workspace_bytes, stream)


def tri_attn_fwd_batched(node, dtype, batch, n, h, d, scale, q, k, v, g, bias, mask, out, lse,
                         workspace, workspace_bytes, stream) -> int:
    """Raw call: every tensor argument is an integer device address (or None)."""
    return lib().tri_attn_fwd_batched(node, dtype, batch, n, h, d, scale, q, k, v, g, bias, mask,
                                      out, lse, workspace, workspace_bytes, stream)


def tri_attn_bwd_batched(node, dtype, batch, n, h, d, scale, q, k, v, g, bias, mask, out, lse,
                         dout, dq, dk, dv, dg, dbias, workspace, workspace_bytes, stream) -> int:
    """Raw call: every tensor argument is an integer device address (or None)."""
    return lib().tri_attn_bwd_batched(node, dtype, batch, n, h, d, scale, q, k, v, g, bias, mask,
                                      out, lse, dout, dq, dk, dv, dg, dbias, workspace,
                                      workspace_bytes, stream)


def _cols_arr(cols):
    return (_i64 * len(cols))(*[int(c) for c in cols])


def tri_ln_linear_fwd(dtype, m, k, cols, eps, x, gamma, beta, w, outs, mean, rstd,
                      stream) -> int:
    """Raw call: tensor arguments are integer device addresses; cols and outs
    are Python sequences (passed as host arrays)."""
    outs_arr = (_vp * len(outs))(*outs)
    return lib().tri_ln_linear_fwd(dtype, m, k, len(cols), _cols_arr(cols), eps, x, gamma, beta,
                                   w, outs_arr, mean, rstd, stream)


def tri_ln_linear_bwd_workspace_bytes(dtype: int, m: int, k: int, cols) -> int:
    out = _sz(0)
    st = lib().tri_ln_linear_bwd_workspace_bytes(dtype, m, k, len(cols), _cols_arr(cols),
                                                 ctypes.byref(out))
    if st != OK:
        raise TriAttnError(st, "tri_ln_linear_bwd_workspace_bytes")
    return out.value


def tri_ln_linear_bwd(dtype, m, k, cols, x, gamma, beta, w, mean, rstd, douts, dx, dw, dgamma,
                      dbeta, workspace, workspace_bytes, stream) -> int:
    """Raw call: tensor arguments are integer device addresses; cols and douts
    are Python sequences (passed as host arrays)."""
    douts_arr = (_vp * len(douts))(*douts)
    return lib().tri_ln_linear_bwd(dtype, m, k, len(cols), _cols_arr(cols), x, gamma, beta, w,
                                   mean, rstd, douts_arr, dx, dw, dgamma, dbeta, workspace,
                                   workspace_bytes, stream)


def tri_transition_fwd_workspace_bytes(dtype: int, m: int, c: int, f: int) -> int:
    out = _sz(0)
    st = lib().tri_transition_fwd_workspace_bytes(dtype, m, c, f, ctypes.byref(out))
    if st != OK:
        raise TriAttnError(st, "tri_transition_fwd_workspace_bytes")
    return out.value


def tri_transition_bwd_workspace_bytes(dtype: int, m: int, c: int, f: int) -> int:
    out = _sz(0)
    st = lib().tri_transition_bwd_workspace_bytes(dtype, m, c, f, ctypes.byref(out))
    if st != OK:
        raise TriAttnError(st, "tri_transition_bwd_workspace_bytes")
    return out.value


def tri_transition_fwd(dtype, m, c, f, eps, x, gamma, beta, w1, w2, out, mean, rstd, workspace,
                       workspace_bytes, stream) -> int:
    """Raw call: every tensor argument is an integer device address (or None)."""
    return lib().tri_transition_fwd(dtype, m, c, f, eps, x, gamma, beta, w1, w2, out, mean,
                                    rstd, workspace, workspace_bytes, stream)


def tri_transition_bwd(dtype, m, c, f, x, gamma, beta, w1, w2, mean, rstd, dout, dx, dw1, dw2,
                       dgamma, dbeta, workspace, workspace_bytes, stream) -> int:
    """Raw call: every tensor argument is an integer device address (or None)."""
    return lib().tri_transition_bwd(dtype, m, c, f, x, gamma, beta, w1, w2, mean, rstd, dout,
                                    dx, dw1, dw2, dgamma, dbeta, workspace, workspace_bytes,
                                    stream)


def tri_attn_timing_enable(on: bool) -> None:
    st = lib().tri_attn_timing_enable(1 if on else 0)
    if st != OK:
        raise TriAttnError(st, "tri_attn_timing_enable")


def tri_attn_timing_select(names=None) -> None:
    """Time only the kernels named in `names` (None: every kernel)."""
    mask = 0
    if names is not None:
        index = {}
        i = 0
        while True:
            r = tri_attn_timing_read(i)
            if r is None:
                break
            index[r[0]] = i
            i += 1
        for n in names:
            if n not in index:
                raise ValueError(f"unknown kernel name {n!r}")
            mask |= 1 << index[n]
    st = lib().tri_attn_timing_select(mask)
    if st != OK:
        raise TriAttnError(st, "tri_attn_timing_select")


def tri_attn_timing_reset() -> None:
    st = lib().tri_attn_timing_reset()
    if st != OK:
        raise TriAttnError(st, "tri_attn_timing_reset")


def tri_attn_timing_read(index: int):
    """(name, total_ms, launches) of kernel `index`, or None past the last one."""
    name, ms, cnt = ctypes.c_char_p(), ctypes.c_double(), ctypes.c_int64()
    st = lib().tri_attn_timing_read(index, ctypes.byref(name), ctypes.byref(ms),
                                    ctypes.byref(cnt))
    if st == ERR_INVALID_ARG:
        return None
    if st != OK:
        raise TriAttnError(st, "tri_attn_timing_read")
    return name.value.decode(), ms.value, cnt.value


def kernel_times():
    """{kernel name: (total ms, launches)} accumulated since the last reset."""
    out, i = {}, 0
    while True:
        r = tri_attn_timing_read(i)
        if r is None:
            return out
        out[r[0]] = (r[1], r[2])
        i += 1


# ---- torch convenience wrappers -------------------------------------------------------

_DTYPES = {torch.float32: F32, torch.bfloat16: BF16}


def _check(name, t, shape, dtype, device):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device != device or t.device.type != "cuda":
        raise ValueError(f"{name} must be on {device} (got {t.device})")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype} (got {t.dtype})")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)} (got {tuple(t.shape)})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _common(q, k, v, g, bias, mask):
    """Shapes of a single map ([n, n, h, d]) or a batch ([b, n, n, h, d]);
    returns (lead, n, h, d, dtype code, device) with lead = () or (b,)."""
    if q.dim() not in (4, 5):
        raise ValueError("q must be [n, n, h, d] or [b, n, n, h, d]")
    lead = tuple(q.shape[:-4])
    n, n2, h, d = q.shape[-4:]
    if n != n2:
        raise ValueError("q must be square in its two pair axes")
    if q.dtype not in _DTYPES:
        raise ValueError(f"unsupported dtype {q.dtype}")
    dev = q.device
    for name, t in (("q", q), ("k", k), ("v", v), ("g", g)):
        _check(name, t, lead + (n, n, h, d), q.dtype, dev)
    _check("bias", bias, lead + (n, n, h), q.dtype, dev)
    if mask is not None:
        _check("mask", mask, lead + (n, n), torch.uint8, dev)
    return lead, n, h, d, _DTYPES[q.dtype], dev


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else t.data_ptr()


def _stream(dev):
    return torch.cuda.current_stream(dev).cuda_stream


# The torch wrappers give a batch one workspace copy per sample (one launch per
# kernel for the whole batch) up to this size, and the unbatched workspace
# (sample by sample) beyond it.
BATCH_WORKSPACE_LIMIT = 4 << 30


def _batch_workspace(batched: int, one: int) -> int:
    return batched if batched <= max(one, BATCH_WORKSPACE_LIMIT) else one


def default_scale(d: int) -> float:
    return 1.0 / math.sqrt(d)


def fwd(q, k, v, g, bias, mask=None, node: int = STARTING, scale: Optional[float] = None,
        workspace: Optional[torch.Tensor] = None):
    """Triangle attention forward.  Returns (out [n,n,h,d], lse [n,n,h] fp32);
    with a leading batch axis on every tensor, the batched call."""
    lead, n, h, d, dt, dev = _common(q, k, v, g, bias, mask)
    scale = default_scale(d) if scale is None else float(scale)
    out = torch.empty_like(q)
    lse = torch.empty(lead + (n, n, h), dtype=torch.float32, device=dev)
    # a batch gets one copy of the workspace per sample (one launch per kernel
    # for the whole batch); a smaller workspace passed in runs it sample by sample
    one = tri_attn_fwd_workspace_bytes(node, dt, n, h, d)
    need = _batch_workspace(tri_attn_fwd_batched_workspace_bytes(node, dt, lead[0], n, h, d),
                            one) if lead else one
    if workspace is None or workspace.numel() < one:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    args = (scale, _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(bias), _ptr(mask), _ptr(out),
            _ptr(lse), _ptr(workspace), workspace.numel(), _stream(dev))
    if lead:
        st = tri_attn_fwd_batched(node, dt, lead[0], n, h, d, *args)
    else:
        st = tri_attn_fwd(node, dt, n, h, d, *args)
    if st != OK:
        raise TriAttnError(st, "tri_attn_fwd_batched" if lead else "tri_attn_fwd")
    return out, lse


def fwd_noalloc(q, k, v, g, bias, mask=None, node: int = STARTING,
                scale: Optional[float] = None, out: Optional[torch.Tensor] = None,
                lse: Optional[torch.Tensor] = None):
    """Triangle attention forward through the allocation-free entry point (the
    library's own scratch array instead of a workspace).  out and lse may be
    passed in; otherwise they are allocated here (the library allocates
    nothing).  Unbatched only."""
    lead, n, h, d, dt, dev = _common(q, k, v, g, bias, mask)
    if lead:
        raise ValueError("fwd_noalloc takes one pair map (no batch axis)")
    scale = default_scale(d) if scale is None else float(scale)
    if out is None:
        out = torch.empty_like(q)
    if lse is None:
        lse = torch.empty((n, n, h), dtype=torch.float32, device=dev)
    _check("out", out, (n, n, h, d), q.dtype, dev)
    _check("lse", lse, (n, n, h), torch.float32, dev)
    st = tri_attn_fwd_noalloc(node, dt, n, h, d, scale, _ptr(q), _ptr(k), _ptr(v), _ptr(g),
                              _ptr(bias), _ptr(mask), _ptr(out), _ptr(lse), _stream(dev))
    if st != OK:
        raise TriAttnError(st, "tri_attn_fwd_noalloc")
    return out, lse


def bwd(q, k, v, g, bias, out, lse, dout, mask=None, node: int = STARTING,
        scale: Optional[float] = None, workspace: Optional[torch.Tensor] = None):
    """Triangle attention backward.  Returns (dq, dk, dv, dg, dbias); batched
    when the tensors have a leading batch axis."""
    lead, n, h, d, dt, dev = _common(q, k, v, g, bias, mask)
    _check("out", out, lead + (n, n, h, d), q.dtype, dev)
    _check("dout", dout, lead + (n, n, h, d), q.dtype, dev)
    _check("lse", lse, lead + (n, n, h), torch.float32, dev)
    scale = default_scale(d) if scale is None else float(scale)
    dq, dk, dv, dg = (torch.empty_like(q) for _ in range(4))
    dbias = torch.empty_like(bias)
    one = tri_attn_bwd_workspace_bytes(node, dt, n, h, d)
    need = _batch_workspace(tri_attn_bwd_batched_workspace_bytes(node, dt, lead[0], n, h, d),
                            one) if lead else one
    if workspace is None or workspace.numel() < one:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    args = (scale, _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(bias), _ptr(mask), _ptr(out),
            _ptr(lse), _ptr(dout), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(dg), _ptr(dbias),
            _ptr(workspace), workspace.numel(), _stream(dev))
    if lead:
        st = tri_attn_bwd_batched(node, dt, lead[0], n, h, d, *args)
    else:
        st = tri_attn_bwd(node, dt, n, h, d, *args)
    if st != OK:
        raise TriAttnError(st, "tri_attn_bwd_batched" if lead else "tri_attn_bwd")
    return dq, dk, dv, dg, dbias


def _rows_common(q, k, v, g, bias, mask):
    if q.dim() != 4:
        raise ValueError("q must be [rows, n, h, d]")
    rows, n, h, d = q.shape
    if q.dtype not in _DTYPES:
        raise ValueError(f"unsupported dtype {q.dtype}")
    dev = q.device
    for name, t in (("q", q), ("k", k), ("v", v), ("g", g)):
        _check(name, t, (rows, n, h, d), q.dtype, dev)
    _check("bias", bias, (n, n, h), q.dtype, dev)
    if mask is not None:
        _check("mask", mask, (rows, n), torch.uint8, dev)
    return rows, n, h, d, _DTYPES[q.dtype], dev


def rows_fwd(q, k, v, g, bias, mask=None, scale: Optional[float] = None,
             workspace: Optional[torch.Tensor] = None):
    """Starting-node forward over a range of rows: q, k, v, g [rows, n, h, d]
    (the range's rows), bias [n, n, h] (whole map), mask [rows, n].  Returns
    (out [rows, n, h, d], lse [rows, n, h] fp32)."""
    rows, n, h, d, dt, dev = _rows_common(q, k, v, g, bias, mask)
    scale = default_scale(d) if scale is None else float(scale)
    out = torch.empty_like(q)
    lse = torch.empty((rows, n, h), dtype=torch.float32, device=dev)
    need = tri_attn_rows_fwd_workspace_bytes(dt, n, rows, h, d)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    st = tri_attn_rows_fwd(dt, n, rows, h, d, scale, _ptr(q), _ptr(k), _ptr(v), _ptr(g),
                           _ptr(bias), _ptr(mask), _ptr(out), _ptr(lse), _ptr(workspace),
                           workspace.numel(), _stream(dev))
    if st != OK:
        raise TriAttnError(st, "tri_attn_rows_fwd")
    return out, lse


def rows_bwd(q, k, v, g, bias, out, lse, dout, mask=None, scale: Optional[float] = None,
             workspace: Optional[torch.Tensor] = None):
    """Starting-node backward over a range of rows.  Returns (dq, dk, dv, dg
    [rows, n, h, d], dbias_partial [n, n, h] fp32: the range's term of the
    bias gradient)."""
    rows, n, h, d, dt, dev = _rows_common(q, k, v, g, bias, mask)
    _check("out", out, (rows, n, h, d), q.dtype, dev)
    _check("dout", dout, (rows, n, h, d), q.dtype, dev)
    _check("lse", lse, (rows, n, h), torch.float32, dev)
    scale = default_scale(d) if scale is None else float(scale)
    dq, dk, dv, dg = (torch.empty_like(q) for _ in range(4))
    dbp = torch.empty((n, n, h), dtype=torch.float32, device=dev)
    need = tri_attn_rows_bwd_workspace_bytes(dt, n, rows, h, d)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    st = tri_attn_rows_bwd(dt, n, rows, h, d, scale, _ptr(q), _ptr(k), _ptr(v), _ptr(g),
                           _ptr(bias), _ptr(mask), _ptr(out), _ptr(lse), _ptr(dout), _ptr(dq),
                           _ptr(dk), _ptr(dv), _ptr(dg), _ptr(dbp), _ptr(workspace),
                           workspace.numel(), _stream(dev))
    if st != OK:
        raise TriAttnError(st, "tri_attn_rows_bwd")
    return dq, dk, dv, dg, dbp


class TriangleAttention(torch.autograd.Function):
    """autograd wrapper: out = triangle_attention(q, k, v, g, bias; mask, node)."""

    @staticmethod
    def forward(ctx, q, k, v, g, bias, mask=None, node=STARTING, scale=None):
        out, lse = fwd(q, k, v, g, bias, mask, node, scale)
        ctx.save_for_backward(q, k, v, g, bias, out, lse)
        ctx.mask, ctx.node, ctx.scale = mask, node, scale
        return out

    @staticmethod
    def backward(ctx, dout):
        q, k, v, g, bias, out, lse = ctx.saved_tensors
        grads = bwd(q, k, v, g, bias, out, lse, dout.contiguous(), ctx.mask, ctx.node, ctx.scale)
        return (*grads, None, None, None)


def triangle_attention(q, k, v, g, bias, mask=None, node: int = STARTING, scale=None):
    return TriangleAttention.apply(q, k, v, g, bias, mask, node, scale)


# ---- fused layer-norm + linear projection ---------------------------------------------

def ln_linear_fwd(x, gamma, beta, w, cols, eps: float = 1e-5):
    """o2 = layer_norm(x) * gamma + beta, then @ w, split column-wise into
    len(cols) tensors [m, cols[i]].  x [m, k] bf16.  Returns (outs, mean,
    rstd)."""
    if x.dim() != 2:
        raise ValueError("x must be [m, k]")
    m, k = x.shape
    dev = x.device
    ncols = int(sum(cols))
    _check("x", x, (m, k), torch.bfloat16, dev)
    _check("gamma", gamma, (k,), torch.bfloat16, dev)
    _check("beta", beta, (k,), torch.bfloat16, dev)
    _check("w", w, (k, ncols), torch.bfloat16, dev)
    outs = [torch.empty((m, int(c)), dtype=torch.bfloat16, device=dev) for c in cols]
    mean = torch.empty(m, dtype=torch.float32, device=dev)
    rstd = torch.empty(m, dtype=torch.float32, device=dev)
    st = tri_ln_linear_fwd(BF16, m, k, cols, float(eps), _ptr(x), _ptr(gamma), _ptr(beta),
                           _ptr(w), [o.data_ptr() for o in outs], _ptr(mean), _ptr(rstd),
                           _stream(dev))
    if st != OK:
        raise TriAttnError(st, "tri_ln_linear_fwd")
    return outs, mean, rstd


def ln_linear_bwd(x, gamma, beta, w, mean, rstd, douts, eps: float = 1e-5,
                  workspace: Optional[torch.Tensor] = None):
    """Gradients of sum(do2 * o2) for ln_linear_fwd: douts are do2 split like
    the forward's outputs.  Returns (dx [m, k] bf16, dw [k, ncols] fp32,
    dgamma [k] fp32, dbeta [k] fp32).  eps is unused (the saved rstd holds it)."""
    m, k = x.shape
    dev = x.device
    cols = [int(d.shape[1]) for d in douts]
    ncols = sum(cols)
    _check("x", x, (m, k), torch.bfloat16, dev)
    _check("gamma", gamma, (k,), torch.bfloat16, dev)
    _check("beta", beta, (k,), torch.bfloat16, dev)
    _check("w", w, (k, ncols), torch.bfloat16, dev)
    _check("mean", mean, (m,), torch.float32, dev)
    _check("rstd", rstd, (m,), torch.float32, dev)
    for i, d in enumerate(douts):
        _check(f"douts[{i}]", d, (m, cols[i]), torch.bfloat16, dev)
    dx = torch.empty_like(x)
    dw = torch.empty((k, ncols), dtype=torch.float32, device=dev)
    dgamma = torch.empty(k, dtype=torch.float32, device=dev)
    dbeta = torch.empty(k, dtype=torch.float32, device=dev)
    need = tri_ln_linear_bwd_workspace_bytes(BF16, m, k, cols)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    st = tri_ln_linear_bwd(BF16, m, k, cols, _ptr(x), _ptr(gamma), _ptr(beta), _ptr(w),
                           _ptr(mean), _ptr(rstd), [d.data_ptr() for d in douts], _ptr(dx),
                           _ptr(dw), _ptr(dgamma), _ptr(dbeta), _ptr(workspace),
                           workspace.numel(), _stream(dev))
    if st != OK:
        raise TriAttnError(st, "tri_ln_linear_bwd")
    return dx, dw, dgamma, dbeta


# ---- fused transition layer -------------------------------------------------------------

def _trn_common(x, gamma, beta, w1, w2):
    if x.dim() != 2:
        raise ValueError("x must be [m, c]")
    m, c = x.shape
    f = w2.shape[0]
    dev = x.device
    _check("x", x, (m, c), torch.bfloat16, dev)
    _check("gamma", gamma, (c,), torch.bfloat16, dev)
    _check("beta", beta, (c,), torch.bfloat16, dev)
    _check("w1", w1, (c, 2 * f), torch.bfloat16, dev)
    _check("w2", w2, (f, c), torch.bfloat16, dev)
    return m, c, f, dev


def transition_fwd(x, gamma, beta, w1, w2, eps: float = 1e-5,
                   workspace: Optional[torch.Tensor] = None):
    """out = (silu(a) * b) @ w2 with [a | b] = layer_norm(x) * gamma + beta
    @ w1.  x [m, c] bf16, w1 [c, 2f], w2 [f, c].  Returns (out, mean, rstd)."""
    m, c, f, dev = _trn_common(x, gamma, beta, w1, w2)
    out = torch.empty_like(x)
    mean = torch.empty(m, dtype=torch.float32, device=dev)
    rstd = torch.empty(m, dtype=torch.float32, device=dev)
    need = tri_transition_fwd_workspace_bytes(BF16, m, c, f)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    st = tri_transition_fwd(BF16, m, c, f, float(eps), _ptr(x), _ptr(gamma), _ptr(beta),
                            _ptr(w1), _ptr(w2), _ptr(out), _ptr(mean), _ptr(rstd),
                            _ptr(workspace), workspace.numel(), _stream(dev))
    if st != OK:
        raise TriAttnError(st, "tri_transition_fwd")
    return out, mean, rstd


def transition_bwd(x, gamma, beta, w1, w2, mean, rstd, dout,
                   workspace: Optional[torch.Tensor] = None):
    """Gradients of sum(dout * out) for transition_fwd.  Returns (dx [m, c]
    bf16, dw1 [c, 2f], dw2 [f, c], dgamma [c], dbeta [c], all fp32 but dx)."""
    m, c, f, dev = _trn_common(x, gamma, beta, w1, w2)
    _check("mean", mean, (m,), torch.float32, dev)
    _check("rstd", rstd, (m,), torch.float32, dev)
    _check("dout", dout, (m, c), torch.bfloat16, dev)
    dx = torch.empty_like(x)
    dw1 = torch.empty((c, 2 * f), dtype=torch.float32, device=dev)
    dw2 = torch.empty((f, c), dtype=torch.float32, device=dev)
    dgamma = torch.empty(c, dtype=torch.float32, device=dev)
    dbeta = torch.empty(c, dtype=torch.float32, device=dev)
    need = tri_transition_bwd_workspace_bytes(BF16, m, c, f)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    st = tri_transition_bwd(BF16, m, c, f, _ptr(x), _ptr(gamma), _ptr(beta), _ptr(w1),
                            _ptr(w2), _ptr(mean), _ptr(rstd), _ptr(dout), _ptr(dx), _ptr(dw1),
                            _ptr(dw2), _ptr(dgamma), _ptr(dbeta), _ptr(workspace),
                            workspace.numel(), _stream(dev))
    if st != OK:
        raise TriAttnError(st, "tri_transition_bwd")
    return dx, dw1, dw2, dgamma, dbeta

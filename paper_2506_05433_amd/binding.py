"""Thin ctypes binding of ``libpg_attn.so`` (argument marshalling only).

Every step of the computation runs in the HIP library; this module only turns
torch device tensors into pointers and sizes, allocates outputs and the
workspace with torch, and passes the current HIP stream. It fails loudly when
the library has not been built: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
# PG_LIB overrides the library file (used to compare builds of the same sources)
LIB_PATH = os.environ.get("PG_LIB") or os.path.join(HERE, "libpg_attn.so")

PG_BF16, PG_FP32 = 0, 1
STATUS = {0: "PG_OK", 1: "PG_EINVAL", 2: "PG_EUNSUPPORTED", 3: "PG_EWORKSPACE", 4: "PG_EHIP"}

_lib = None

# names and argument types of every function include/pg_attn.h declares
_I, _Z, _F, _P = ctypes.c_int, ctypes.c_size_t, ctypes.c_float, ctypes.c_void_p
SIGNATURES = {
    "pg_attn_fwd_workspace_size": (_Z, [_I, _I, _I, _I, _I, _I, _I]),
    "pg_attn_bwd_workspace_size": (_Z, [_I, _I, _I, _I, _I, _I, _I]),
    "pg_attn_fwd": (_I, [_I, _I, _I, _I, _I, _P, _P, _P, _I, _I, _I, _F] + [_P] * 10 + [_P, _Z, _P]),
    "pg_attn_bwd": (_I, [_I, _I, _I, _I, _I, _P, _P, _P, _I, _I, _I, _F] + [_P] * 18 + [_P, _Z, _P]),
    "pg_attn_fwd_noalloc": (_I, [_I, _I, _I, _I, _I, _P, _P, _P, _I, _I, _I, _F] + [_P] * 10 + [_P]),
    "pg_attn_fwd_xours": (_I, [_I, _I, _I, _I, _I, _P, _P, _P, _I, _I, _I, _F] + [_P] * 5 + [_P, _Z, _P]),
    "pg_attn_bwd_xours": (_I, [_I, _I, _I, _I, _I, _P, _P, _P, _I, _I, _I, _F] + [_P] * 9 + [_P, _Z, _P]),
    "pg_attn_fwd_last_workspace_size": (_Z, [_I, _I, _I, _I, _I, _I, _I]),
    "pg_attn_fwd_last": (_I, [_I, _I, _I, _I, _I, _P, _P, _P, _I, _I, _I, _F] + [_P] * 8 + [_P, _Z, _P]),
    "pg_rope_workspace_size": (_Z, [_I]),
    "pg_rope": (_I, [_I, _I, _I, _I, _I, _P, _P, _P, _I, _I, _I, _I, ctypes.c_double, _I] + [_P] * 8 + [_P, _Z, _P]),
    "pg_grouped_positions": (_I, [_I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _Z, _P]),
    "pg_timing_start": (_I, []),
    "pg_timing_stop": (_I, []),
    "pg_timing_get": (_I, [_I, ctypes.POINTER(ctypes.c_int), ctypes.POINTER(ctypes.c_double)]),
    "pg_plan_status": (_I, [_P, _Z, _P]),
    "pg_status_string": (ctypes.c_char_p, [_I]),
    "pg_last_error": (ctypes.c_char_p, []),
}


class PgError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status


def lib():
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2506_05433_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


KERNELS = {"plan": 0, "fwd": 1, "dkdv": 3, "dq": 4, "rope": 5, "last": 6, "kv_reduce": 7}
ROPE_INVERSE, ROPE_INTERLEAVED = 1, 2


def timing_start():
    _check(lib().pg_timing_start())


def timing_stop():
    _check(lib().pg_timing_stop())


def timing_get(kernel: str):
    """(launches, total_ms) recorded for one kernel kind since timing_start()."""
    n, ms = ctypes.c_int(0), ctypes.c_double(0.0)
    _check(lib().pg_timing_get(KERNELS[kernel], ctypes.byref(n), ctypes.byref(ms)))
    return n.value, ms.value


def _check(status: int):
    if status != 0:
        raise PgError(status, lib().pg_last_error().decode())


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _dtype_code(torch, dt):
    if dt == torch.bfloat16:
        return PG_BF16
    if dt == torch.float32:
        return PG_FP32
    raise TypeError(f"unsupported dtype {dt}")


def _stream(torch, device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def workspace_bytes(kind: str, n_groups, n_suffixes, total_prefix, total_suffix, h_q, h_kv, head_dim) -> int:
    fn = lib().pg_attn_fwd_workspace_size if kind == "fwd" else lib().pg_attn_bwd_workspace_size
    return int(fn(n_groups, n_suffixes, total_prefix, total_suffix, h_q, h_kv, head_dim))


def _shapes(q_pre, k_pre, q_suf, cu_prefix, cu_suffix, group_sizes):
    n_groups = group_sizes.numel()
    n_suffixes = cu_suffix.numel() - 1
    if cu_prefix.numel() != n_groups + 1:
        raise ValueError("cu_prefix_lens must have n_groups + 1 entries")
    for t in (cu_prefix, cu_suffix, group_sizes):
        if t.dtype.itemsize != 4 or t.dtype.is_floating_point or not t.is_contiguous():
            raise TypeError("grouping arrays must be contiguous int32 device tensors")
    if q_pre.dim() != 3 or q_suf.dim() != 3 or k_pre.dim() != 3:
        raise ValueError("q and k tensors must be [rows, heads, head_dim]")
    return n_groups, n_suffixes, q_pre.shape[0], q_suf.shape[0], q_pre.shape[1], k_pre.shape[1], q_pre.shape[2]


def _expect(device, dtype, **tensors):
    """Every named tensor is (shape, tensor): contiguous, of that shape, dtype (None: float32) and device.

    The library receives raw pointers, so a strided view, a wrong shape or a tensor on another device would
    be read or written out of place; they are rejected here instead."""
    import torch
    for name, (shape, t) in tensors.items():
        want = torch.float32 if dtype is None or name.startswith("lse") else dtype
        if not isinstance(t, torch.Tensor):
            raise TypeError(f"{name} must be a tensor")
        if tuple(t.shape) != tuple(shape):
            raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
        if t.dtype != want:
            raise TypeError(f"{name} has dtype {t.dtype}, expected {want}")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
        if t.device != device:
            raise ValueError(f"{name} is on {t.device}, expected {device}")
    if device.type != "cuda":
        raise ValueError(f"tensors must be GPU device memory, got {device}")


def _workspace(t, device):
    import torch
    if t.dtype != torch.uint8 or not t.is_contiguous() or t.device != device:
        raise ValueError("workspace must be a contiguous uint8 tensor on the tensors' device")


def fwd(q_pre, k_pre, v_pre, q_suf, k_suf, v_suf, cu_prefix, cu_suffix, group_sizes, scale,
        out=None, workspace=None):
    """Grouped attention forward. Returns (o_pre, o_suf, lse_pre, lse_suf)."""
    import torch
    ng, ns, tp, ts, hq, hkv, d = _shapes(q_pre, k_pre, q_suf, cu_prefix, cu_suffix, group_sizes)
    dev, dt = q_pre.device, q_pre.dtype
    if out is None:
        out = (torch.empty_like(q_pre), torch.empty_like(q_suf),
               torch.empty((hq, tp), device=dev, dtype=torch.float32),
               torch.empty((hq, ts), device=dev, dtype=torch.float32))
    need = workspace_bytes("fwd", ng, ns, tp, ts, hq, hkv, d)
    if workspace is None:
        workspace = torch.empty(need, device=dev, dtype=torch.uint8)
    o_pre, o_suf, lse_pre, lse_suf = out
    _expect(dev, dt, q_pre=((tp, hq, d), q_pre), k_pre=((tp, hkv, d), k_pre), v_pre=((tp, hkv, d), v_pre),
            q_suf=((ts, hq, d), q_suf), k_suf=((ts, hkv, d), k_suf), v_suf=((ts, hkv, d), v_suf),
            o_pre=((tp, hq, d), o_pre), o_suf=((ts, hq, d), o_suf), lse_pre=((hq, tp), lse_pre),
            lse_suf=((hq, ts), lse_suf))
    _workspace(workspace, dev)
    st = lib().pg_attn_fwd(
        _dtype_code(torch, q_pre.dtype), ng, ns, tp, ts,
        _ptr(cu_prefix), _ptr(cu_suffix), _ptr(group_sizes), hq, hkv, d, float(scale),
        _ptr(q_pre), _ptr(k_pre), _ptr(v_pre), _ptr(q_suf), _ptr(k_suf), _ptr(v_suf),
        _ptr(o_pre), _ptr(o_suf), _ptr(lse_pre), _ptr(lse_suf),
        _ptr(workspace), workspace.numel() * workspace.element_size(), _stream(torch, dev))
    _check(st)
    return o_pre, o_suf, lse_pre, lse_suf


def bwd(q_pre, k_pre, v_pre, q_suf, k_suf, v_suf, o_pre, o_suf, lse_pre, lse_suf, do_pre, do_suf,
        cu_prefix, cu_suffix, group_sizes, scale, out=None, workspace=None):
    """Grouped attention backward. Returns (dq_pre, dk_pre, dv_pre, dq_suf, dk_suf, dv_suf)."""
    import torch
    ng, ns, tp, ts, hq, hkv, d = _shapes(q_pre, k_pre, q_suf, cu_prefix, cu_suffix, group_sizes)
    dev, dt = q_pre.device, q_pre.dtype
    if out is None:
        out = (torch.empty_like(q_pre), torch.empty_like(k_pre), torch.empty_like(v_pre),
               torch.empty_like(q_suf), torch.empty_like(k_suf), torch.empty_like(v_suf))
    need = workspace_bytes("bwd", ng, ns, tp, ts, hq, hkv, d)
    if workspace is None:
        workspace = torch.empty(need, device=dev, dtype=torch.uint8)
    pre_q, pre_kv, suf_q, suf_kv = (tp, hq, d), (tp, hkv, d), (ts, hq, d), (ts, hkv, d)
    _expect(dev, dt, q_pre=(pre_q, q_pre), k_pre=(pre_kv, k_pre), v_pre=(pre_kv, v_pre), q_suf=(suf_q, q_suf),
            k_suf=(suf_kv, k_suf), v_suf=(suf_kv, v_suf), o_pre=(pre_q, o_pre), o_suf=(suf_q, o_suf),
            lse_pre=((hq, tp), lse_pre), lse_suf=((hq, ts), lse_suf), do_pre=(pre_q, do_pre),
            do_suf=(suf_q, do_suf), dq_pre=(pre_q, out[0]), dk_pre=(pre_kv, out[1]), dv_pre=(pre_kv, out[2]),
            dq_suf=(suf_q, out[3]), dk_suf=(suf_kv, out[4]), dv_suf=(suf_kv, out[5]))
    _workspace(workspace, dev)
    st = lib().pg_attn_bwd(
        _dtype_code(torch, q_pre.dtype), ng, ns, tp, ts,
        _ptr(cu_prefix), _ptr(cu_suffix), _ptr(group_sizes), hq, hkv, d, float(scale),
        _ptr(q_pre), _ptr(k_pre), _ptr(v_pre), _ptr(q_suf), _ptr(k_suf), _ptr(v_suf),
        _ptr(o_pre), _ptr(o_suf), _ptr(lse_pre), _ptr(lse_suf), _ptr(do_pre), _ptr(do_suf),
        *[_ptr(t) for t in out],
        _ptr(workspace), workspace.numel() * workspace.element_size(), _stream(torch, dev))
    _check(st)
    return out


def plan_status(workspace=None):
    """Raise PgError(PG_EINVAL) if the last call that used ``workspace`` (None: the last pg_attn_fwd_noalloc on
    the current device) found its grouping arrays inconsistent; waits for the current stream."""
    import torch
    if workspace is None:
        st = lib().pg_plan_status(None, 0, _stream(torch, torch.device("cuda", torch.cuda.current_device())))
    else:
        st = lib().pg_plan_status(_ptr(workspace), workspace.numel(), _stream(torch, workspace.device))
    _check(st)


def fwd_noalloc(q_pre, k_pre, v_pre, q_suf, k_suf, v_suf, cu_prefix, cu_suffix, group_sizes, scale, out):
    """Forward without a workspace (pg_attn_fwd_noalloc): the plan lives in the library's per-device scratch
    array. ``out`` = (o_pre, o_suf, lse_pre, lse_suf), preallocated by the caller. Returns ``out``."""
    import torch
    ng, ns, tp, ts, hq, hkv, d = _shapes(q_pre, k_pre, q_suf, cu_prefix, cu_suffix, group_sizes)
    dev, dt = q_pre.device, q_pre.dtype
    o_pre, o_suf, lse_pre, lse_suf = out
    _expect(dev, dt, q_pre=((tp, hq, d), q_pre), k_pre=((tp, hkv, d), k_pre), v_pre=((tp, hkv, d), v_pre),
            q_suf=((ts, hq, d), q_suf), k_suf=((ts, hkv, d), k_suf), v_suf=((ts, hkv, d), v_suf),
            o_pre=((tp, hq, d), o_pre), o_suf=((ts, hq, d), o_suf), lse_pre=((hq, tp), lse_pre),
            lse_suf=((hq, ts), lse_suf))
    st = lib().pg_attn_fwd_noalloc(
        _dtype_code(torch, dt), ng, ns, tp, ts,
        _ptr(cu_prefix), _ptr(cu_suffix), _ptr(group_sizes), hq, hkv, d, float(scale),
        _ptr(q_pre), _ptr(k_pre), _ptr(v_pre), _ptr(q_suf), _ptr(k_suf), _ptr(v_suf),
        _ptr(o_pre), _ptr(o_suf), _ptr(lse_pre), _ptr(lse_suf), _stream(torch, dev))
    _check(st)
    return out


def fwd_xours(q, k, v, cu_prefix, cu_suffix, group_sizes, total_prefix, scale, out=None, workspace=None):
    """Forward on the single-buffer layout of Eq. (2) (pg_attn_fwd_xours): q [rows, h_q, d], k, v
    [rows, h_kv, d], rows grouped as [P; R_1; ...; R_G] per group. Returns (o, lse [h_q, rows])."""
    import torch
    ng, ns = group_sizes.numel(), cu_suffix.numel() - 1
    rows, hq, d = q.shape
    hkv = k.shape[1]
    tp, ts = int(total_prefix), rows - int(total_prefix)
    if out is None:
        out = (torch.empty_like(q), torch.empty((hq, rows), device=q.device, dtype=torch.float32))
    if workspace is None:
        workspace = torch.empty(workspace_bytes("fwd", ng, ns, tp, ts, hq, hkv, d), device=q.device,
                                dtype=torch.uint8)
    o, lse = out
    _expect(q.device, q.dtype, q=((rows, hq, d), q), k=((rows, hkv, d), k), v=((rows, hkv, d), v),
            o=((rows, hq, d), o), lse=((hq, rows), lse))
    _workspace(workspace, q.device)
    st = lib().pg_attn_fwd_xours(_dtype_code(torch, q.dtype), ng, ns, tp, ts, _ptr(cu_prefix), _ptr(cu_suffix),
                                 _ptr(group_sizes), hq, hkv, d, float(scale), _ptr(q), _ptr(k), _ptr(v), _ptr(o),
                                 _ptr(lse), _ptr(workspace), workspace.numel(), _stream(torch, q.device))
    _check(st)
    return o, lse


def bwd_xours(q, k, v, o, lse, d_o, cu_prefix, cu_suffix, group_sizes, total_prefix, scale, out=None,
              workspace=None):
    """Backward on the single-buffer layout (pg_attn_bwd_xours). Returns (dq, dk, dv) in that layout."""
    import torch
    ng, ns = group_sizes.numel(), cu_suffix.numel() - 1
    rows, hq, d = q.shape
    hkv = k.shape[1]
    tp, ts = int(total_prefix), rows - int(total_prefix)
    if out is None:
        out = (torch.empty_like(q), torch.empty_like(k), torch.empty_like(v))
    if workspace is None:
        workspace = torch.empty(workspace_bytes("bwd", ng, ns, tp, ts, hq, hkv, d), device=q.device,
                                dtype=torch.uint8)
    _expect(q.device, q.dtype, q=((rows, hq, d), q), k=((rows, hkv, d), k), v=((rows, hkv, d), v),
            o=((rows, hq, d), o), lse=((hq, rows), lse), d_o=((rows, hq, d), d_o), dq=((rows, hq, d), out[0]),
            dk=((rows, hkv, d), out[1]), dv=((rows, hkv, d), out[2]))
    _workspace(workspace, q.device)
    st = lib().pg_attn_bwd_xours(_dtype_code(torch, q.dtype), ng, ns, tp, ts, _ptr(cu_prefix), _ptr(cu_suffix),
                                 _ptr(group_sizes), hq, hkv, d, float(scale), _ptr(q), _ptr(k), _ptr(v), _ptr(o),
                                 _ptr(lse), _ptr(d_o), *[_ptr(t) for t in out], _ptr(workspace),
                                 workspace.numel(), _stream(torch, q.device))
    _check(st)
    return out


def fwd_last(q_pre, k_pre, v_pre, q_suf, k_suf, v_suf, cu_prefix, cu_suffix, group_sizes, scale, out=None,
             workspace=None):
    """Final-token forward (pg_attn_fwd_last). Returns (o_last [n_suffixes, h_q, d], lse_last [h_q, n_suffixes])."""
    import torch
    ng, ns, tp, ts, hq, hkv, d = _shapes(q_pre, k_pre, q_suf, cu_prefix, cu_suffix, group_sizes)
    dev = q_pre.device
    if out is None:
        out = (torch.empty((ns, hq, d), device=dev, dtype=q_pre.dtype),
               torch.empty((hq, ns), device=dev, dtype=torch.float32))
    if workspace is None:
        nbytes = int(lib().pg_attn_fwd_last_workspace_size(ng, ns, tp, ts, hq, hkv, d))
        workspace = torch.empty(nbytes, device=dev, dtype=torch.uint8)
    o, lse = out
    _expect(dev, q_pre.dtype, q_pre=((tp, hq, d), q_pre), k_pre=((tp, hkv, d), k_pre), v_pre=((tp, hkv, d), v_pre),
            q_suf=((ts, hq, d), q_suf), k_suf=((ts, hkv, d), k_suf), v_suf=((ts, hkv, d), v_suf),
            o_last=((ns, hq, d), o), lse_last=((hq, ns), lse))
    _workspace(workspace, dev)
    st = lib().pg_attn_fwd_last(_dtype_code(torch, q_pre.dtype), ng, ns, tp, ts, _ptr(cu_prefix), _ptr(cu_suffix),
                                _ptr(group_sizes), hq, hkv, d, float(scale), _ptr(q_pre), _ptr(k_pre), _ptr(v_pre),
                                _ptr(q_suf), _ptr(k_suf), _ptr(v_suf), _ptr(o), _ptr(lse), _ptr(workspace),
                                workspace.numel(), _stream(torch, dev))
    _check(st)
    return o, lse


def rope(q_pre, q_suf, k_pre, k_suf, cu_prefix, cu_suffix, group_sizes, base=10000.0, rotary_dim=None,
         inverse=False, interleaved=False, out=None, workspace=None):
    """Rotary embedding with grouped positions (pg_rope). q_* [rows, h_q, d], k_* [rows, h_kv, d]; either
    pair may be None to rotate only the other. ``out`` = (q_pre, q_suf, k_pre, k_suf) destinations (may be
    the inputs themselves); new tensors by default. Returns the four outputs (None where not rotated)."""
    import torch
    ref = q_pre if q_pre is not None else k_pre
    ng, ns = group_sizes.numel(), cu_suffix.numel() - 1
    tp = ref.shape[0]
    ts = (q_suf if q_suf is not None else k_suf).shape[0]
    d = ref.shape[2]
    hq = q_pre.shape[1] if q_pre is not None else 0
    hkv = k_pre.shape[1] if k_pre is not None else 0
    ins = (q_pre, q_suf, k_pre, k_suf)
    if out is None:
        out = tuple(None if t is None else torch.empty_like(t) for t in ins)
    if workspace is None:
        workspace = torch.empty(int(lib().pg_rope_workspace_size(ng)), device=ref.device, dtype=torch.uint8)
    named = {}
    for name, t, o, rows_, h in (("q_pre", q_pre, out[0], tp, hq), ("q_suf", q_suf, out[1], ts, hq),
                                 ("k_pre", k_pre, out[2], tp, hkv), ("k_suf", k_suf, out[3], ts, hkv)):
        if t is not None:
            named[name] = ((rows_, h, d), t)
            named[name + "_out"] = ((rows_, h, d), o)
    _expect(ref.device, ref.dtype, **named)
    _workspace(workspace, ref.device)
    flags = (ROPE_INVERSE if inverse else 0) | (ROPE_INTERLEAVED if interleaved else 0)
    st = lib().pg_rope(_dtype_code(torch, ref.dtype), ng, ns, tp, ts, _ptr(cu_prefix), _ptr(cu_suffix),
                       _ptr(group_sizes), hq, hkv, d, d if rotary_dim is None else int(rotary_dim), float(base),
                       flags, *[_ptr(t) for t in ins], *[_ptr(t) for t in out],
                       _ptr(workspace), workspace.numel(), _stream(torch, ref.device))
    _check(st)
    return out


def grouped_positions(total_prefix, total_suffix, cu_prefix, cu_suffix, group_sizes, workspace=None):
    """(pos_pre, pos_suf) int32 device tensors of the grouped position ids (pg_grouped_positions)."""
    import torch
    dev = cu_suffix.device
    ng, ns = group_sizes.numel(), cu_suffix.numel() - 1
    pos_pre = torch.empty(total_prefix, device=dev, dtype=torch.int32)
    pos_suf = torch.empty(total_suffix, device=dev, dtype=torch.int32)
    if workspace is None:
        workspace = torch.empty(int(lib().pg_rope_workspace_size(ng)), device=dev, dtype=torch.uint8)
    st = lib().pg_grouped_positions(ng, ns, total_prefix, total_suffix, _ptr(cu_prefix), _ptr(cu_suffix),
                                    _ptr(group_sizes), _ptr(pos_pre), _ptr(pos_suf), _ptr(workspace),
                                    workspace.numel(), _stream(torch, dev))
    _check(st)
    return pos_pre, pos_suf


def to_device(prob, device="cuda"):
    """Copy a seeded problem (``paper_2506_05433_amd.inputs.Problem``) to device tensors.

    Returns a dict with the eight tensors (bfloat16 or float32), the int32
    grouping arrays ``cu_prefix``, ``cu_suffix``, ``group_sizes`` and ``scale``.
    """
    import numpy as np
    import torch
    out = {}
    for name, a in prob.tensors.items():
        if a.dtype == np.uint16:
            t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16)
        else:
            t = torch.from_numpy(np.ascontiguousarray(a))
        out[name] = t.to(device)
    out["cu_prefix"] = torch.from_numpy(prob.cu_prefix.astype(np.int32)).to(device)
    out["cu_suffix"] = torch.from_numpy(prob.cu_suffix.astype(np.int32)).to(device)
    out["group_sizes"] = torch.from_numpy(prob.group_sizes.astype(np.int32)).to(device)
    out["scale"] = prob.scale
    return out


def run_fwd(dev):
    """Forward on a ``to_device`` dict."""
    return fwd(dev["q_pre"], dev["k_pre"], dev["v_pre"], dev["q_suf"], dev["k_suf"], dev["v_suf"],
               dev["cu_prefix"], dev["cu_suffix"], dev["group_sizes"], dev["scale"])


def run_bwd(dev, fwd_out):
    """Backward on a ``to_device`` dict and the forward's outputs."""
    o_pre, o_suf, lse_pre, lse_suf = fwd_out
    return bwd(dev["q_pre"], dev["k_pre"], dev["v_pre"], dev["q_suf"], dev["k_suf"], dev["v_suf"],
               o_pre, o_suf, lse_pre, lse_suf, dev["do_pre"], dev["do_suf"],
               dev["cu_prefix"], dev["cu_suffix"], dev["group_sizes"], dev["scale"])

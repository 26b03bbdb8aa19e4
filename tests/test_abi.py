"""C-ABI checks that need no GPU: the library loads, exports every declared
symbol, sizes its workspace, and rejects bad arguments on the host before
anything is launched."""
import ctypes
import os
import re

import pytest

from paper_2506_05433_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pg_attn.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pg_[a-z_0-9]+)\s*\(", text)))


def test_header_declares_the_expected_entry_points():
    assert set(declared_functions()) == set(binding.SIGNATURES)


def test_library_exports_every_declared_symbol():
    L = binding.lib()
    for name in declared_functions():
        assert hasattr(L, name), name


def test_status_strings():
    L = binding.lib()
    for s, tag in binding.STATUS.items():
        assert L.pg_status_string(s).decode().startswith(tag)


def test_workspace_sizes_grow_with_the_problem():
    f1 = binding.workspace_bytes("fwd", 1, 8, 4096, 5120, 32, 8, 128)
    b1 = binding.workspace_bytes("bwd", 1, 8, 4096, 5120, 32, 8, 128)
    f2 = binding.workspace_bytes("fwd", 8, 128, 73275, 266240, 64, 8, 128)
    assert 0 < f1 < b1 and f1 < f2
    # the backward workspace holds rowsum(dO*O): h_q * rows floats
    assert b1 >= 32 * (4096 + 5120) * 4
    assert binding.workspace_bytes("fwd", -1, 0, 0, 0, 1, 1, 64) == 0


def _call_fwd(**over):
    args = dict(dtype=0, ng=1, ns=2, tp=8, ts=6, cu_p=1, cu_s=1, gsz=1, h_q=4, h_kv=2, d=128, scale=0.125,
                ptr=1, ws=1, ws_bytes=1 << 30)
    args.update(over)
    p = lambda v: ctypes.c_void_p(v) if v else None  # noqa: E731
    L = binding.lib()
    return L.pg_attn_fwd(args["dtype"], args["ng"], args["ns"], args["tp"], args["ts"],
                         p(args["cu_p"]), p(args["cu_s"]), p(args["gsz"]), args["h_q"], args["h_kv"], args["d"],
                         args["scale"], *[p(args["ptr"])] * 10, p(args["ws"]), args["ws_bytes"], None)


@pytest.mark.parametrize("over,status", [
    (dict(dtype=7), 2),
    (dict(d=96), 2),
    (dict(h_q=1024, h_kv=2), 2),
    (dict(h_q=6, h_kv=4), 1),
    (dict(h_kv=0), 1),
    (dict(scale=float("nan")), 1),
    (dict(scale=-1.0), 1),
    (dict(tp=-3), 1),
    (dict(ng=0), 1),
    (dict(ns=0), 1),
    (dict(cu_p=0), 1),
    (dict(cu_s=0), 1),
    (dict(ptr=0), 1),
    (dict(ws=0), 3),
    (dict(ws_bytes=16), 3),
])
def test_host_validation_rejects_before_launch(over, status):
    """Bad arguments are rejected on the host (no pointer is dereferenced, nothing launches)."""
    assert _call_fwd(**over) == status
    assert binding.lib().pg_last_error().decode() != ""


def test_bwd_validation():
    L = binding.lib()
    p = ctypes.c_void_p(1)
    st = L.pg_attn_bwd(0, 1, 2, 8, 6, p, p, p, 4, 2, 64, 0.125, *[p] * 18, p, 16, None)
    assert st == 3


def test_valid_call_without_a_gpu_reports_hip_error():
    """With no usable device the call fails with PG_EHIP instead of crashing (host-forced failure path)."""
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    assert _call_fwd() == 4
    assert "hip" in binding.lib().pg_last_error().decode().lower()


def _call_rope(**over):
    args = dict(dtype=0, ng=1, ns=2, tp=8, ts=6, cu=16, h_q=4, h_kv=2, d=128, rot=128, base=10000.0, flags=0,
                ptr=256, ws=256, ws_bytes=1 << 20)
    args.update(over)
    p = lambda v: ctypes.c_void_p(v) if v else None  # noqa: E731
    L = binding.lib()
    return L.pg_rope(args["dtype"], args["ng"], args["ns"], args["tp"], args["ts"], p(args["cu"]), p(args["cu"]),
                     p(args["cu"]), args["h_q"], args["h_kv"], args["d"], args["rot"], args["base"], args["flags"],
                     *[p(args["ptr"])] * 8, p(args["ws"]), args["ws_bytes"], None)


@pytest.mark.parametrize("over,status", [
    (dict(dtype=3), 2),
    (dict(d=96, rot=96), 2),
    (dict(rot=8), 2),
    (dict(rot=40), 2),
    (dict(d=64, rot=128), 2),
    (dict(h_q=0, h_kv=0), 1),
    (dict(h_q=600, h_kv=0), 2),
    (dict(base=0.0), 1),
    (dict(base=float("inf")), 1),
    (dict(flags=4), 1),
    (dict(ptr=0), 1),
    (dict(ptr=264), 1),          # not 16-byte aligned
    (dict(cu=0), 1),
    (dict(ng=0), 1),
    (dict(ws=0), 3),
    (dict(ws_bytes=8), 3),
])
def test_rope_host_validation(over, status):
    assert _call_rope(**over) == status
    assert binding.lib().pg_last_error().decode() != ""


def test_rope_workspace_and_positions_validation():
    L = binding.lib()
    assert L.pg_rope_workspace_size(1) > 0 and L.pg_rope_workspace_size(1000) > L.pg_rope_workspace_size(1)
    assert L.pg_rope_workspace_size(-1) == 0
    p = ctypes.c_void_p(256)
    assert L.pg_grouped_positions(1, 2, 8, 6, p, p, p, None, p, p, 1 << 20, None) == 1   # NULL pos_pre
    assert L.pg_grouped_positions(1, 2, 8, 6, p, p, p, p, p, p, 8, None) == 3            # workspace too small


def test_rope_without_a_gpu_reports_hip_error():
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    assert _call_rope() == 4


def test_xours_validation():
    L = binding.lib()
    p = ctypes.c_void_p(256)
    # a NULL tensor is rejected before launch; a short workspace too
    assert L.pg_attn_fwd_xours(0, 1, 2, 8, 6, p, p, p, 4, 2, 128, 0.125, p, p, None, p, p, p, 1 << 30, None) == 1
    assert L.pg_attn_bwd_xours(0, 1, 2, 8, 6, p, p, p, 4, 2, 128, 0.125, *[p] * 9, p, 16, None) == 3


def test_last_validation_and_workspace():
    L = binding.lib()
    p = ctypes.c_void_p(256)
    assert L.pg_attn_fwd_last_workspace_size(1, 16, 16384, 5000, 32, 8, 128) > 0
    assert L.pg_attn_fwd_last_workspace_size(-1, 16, 0, 0, 32, 8, 128) == 0
    # NULL output, bad head_dim, GQA ratio above 128, short workspace
    assert L.pg_attn_fwd_last(0, 1, 2, 8, 6, p, p, p, 4, 2, 128, 0.125, *[p] * 6, None, p, p, 1 << 30, None) == 1
    assert L.pg_attn_fwd_last(0, 1, 2, 8, 6, p, p, p, 4, 2, 96, 0.125, *[p] * 8, p, 1 << 30, None) == 2
    assert L.pg_attn_fwd_last(0, 1, 2, 8, 6, p, p, p, 256, 1, 128, 0.125, *[p] * 8, p, 1 << 30, None) == 2
    assert L.pg_attn_fwd_last(0, 1, 2, 8, 6, p, p, p, 4, 2, 128, 0.125, *[p] * 8, p, 16, None) == 3


def test_noalloc_forward_rejects_plans_beyond_its_scratch():
    """A plan larger than the scratch array is refused on the host, before any device call."""
    L = binding.lib()
    p = ctypes.c_void_p(1)
    ts = 5_000_000  # the per-row member table alone needs 20 MB
    st = L.pg_attn_fwd_noalloc(0, 1, 1, 0, ts, p, p, p, 1, 1, 64, 0.125, *[p] * 10, None)
    assert st == 2 and b"scratch" in L.pg_last_error()

"""The device planner compiled for the host (tests/host_plan) under AddressSanitizer.

* Inconsistent grouping arrays, including group sizes whose 32-bit sum wraps around to
  n_suffixes, are flagged and never make the planner read past an array.
* Valid arrays: the one-block and the multi-kernel planners give the same plan, and the
  plan is the tiling the kernels assume (prefix tiles of every group, response rows of
  every group stacked into tiles, per-tile member bounds, longest-first order).
* Every load the attention kernels derive from the plan (key/value tiles of the forward
  and dQ kernels, query tiles of the dK/dV walks, per-row tables) stays inside its tensor
  and inside a 2^31-byte buffer range, for the five workloads and the Fig. 2/3 grid.
"""
import math
import os
import shutil
import subprocess

import numpy as np
import pytest

from paper_2506_05433_amd.inputs import WORKLOADS, Workload, draw_lengths

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "host_plan")
CSRC = os.path.join(ROOT, "paper_2506_05433_amd", "csrc")
BM, BKV = 128, 128           # query rows per forward/dQ tile, keys per dK/dV workgroup
BN = 64                      # keys per forward/dQ key tile
BQ = {"bf16": 64, "fp32": 32}  # query rows per dK/dV query tile


@pytest.fixture(scope="module")
def planner(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    exe = str(tmp_path_factory.mktemp("plan") / "plan_host")
    cmd = [gxx, "-std=c++20", "-O1", "-g", "-fsanitize=address,undefined", "-fno-omit-frame-pointer",
           "-fno-sanitize-recover=undefined", "-pthread", "-I", HERE, "-I", CSRC,
           os.path.join(HERE, "plan_host.cpp"), "-o", exe]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-4000:]
    return exe


def kv_chunks_for(ng, tp, ts, h_q, h_kv):
    """The library's split of long prefix key walks (pg_attn.hip, kv_chunks_for)."""
    if tp <= 0 or h_kv <= 0:
        return 1
    tiles = (math.ceil(tp / BKV) + ng) * h_kv
    c = math.ceil(512 / tiles)
    walk = math.ceil((tp + ts) / (max(ng, 1) * 64)) * (h_q // h_kv)
    c = min(c, walk // (1 if 2 * tiles <= 256 else 16))
    return max(1, min(8, c))


def split_for(ng, tp, ts, h_q):
    """The library's choice of member-aligned response tiles (pg_attn.hip, make_layout)."""
    return int((math.ceil(tp / BM) + math.ceil(ts / BM) + ng) * h_q < 256)


def bounds(ng, ns, tp, ts, kvc):
    return (math.ceil(tp / BM) + math.ceil(ts / BM) + 2 * ng + ns,
            (math.ceil(tp / BKV) + ng) * kvc + math.ceil(ts / BKV) + ng + ns)


def run_plan(exe, cu_p, cu_s, gsz, ng, ns, tp, ts, mode=0, kvc=1, split=0, max_q=None, max_kv=None):
    bq, bkv = bounds(ng, ns, tp, ts, kvc)
    max_q = bq if max_q is None else max_q
    max_kv = bkv if max_kv is None else max_kv
    text = " ".join(str(int(x)) for x in [mode, ng, ns, tp, ts, BM, BKV, kvc, split, max_q, max_kv, *cu_p, *cu_s,
                                           *gsz])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0", UBSAN_OPTIONS="halt_on_error=1")
    res = subprocess.run([exe], input=text, capture_output=True, text=True, env=env, timeout=300)
    assert res.returncode == 0, res.stderr[-4000:]
    assert "ERROR: AddressSanitizer" not in res.stderr and "runtime error" not in res.stderr, res.stderr[-4000:]
    lines = res.stdout.split("\n")
    err, nq, nkv = (int(x) for x in lines[0].split())
    q = [tuple(int(x) for x in ln.split()[1:]) for ln in lines[1:] if ln.startswith("q ")]
    k = [tuple(int(x) for x in ln.split()[1:]) for ln in lines[1:] if ln.startswith("k ")]
    s = [ln for ln in lines if ln.startswith("s")]
    seg = [int(x) for x in s[0].split()[1:]] if s else []
    return err, q, k, seg


def arrays(prefix, groups, suffix):
    cu_p = np.concatenate([[0], np.cumsum(prefix)]).astype(np.int64)
    cu_s = np.concatenate([[0], np.cumsum(suffix)]).astype(np.int64)
    return cu_p, cu_s, np.asarray(groups, np.int64)


@pytest.mark.parametrize("gsz,ns", [
    # 32-bit sums that wrap around to n_suffixes (the planner would then index cu_suffix_lens with
    # member starts near 2^31)
    ([0x7FFFFFFF, 0x7FFFFFFF, 2], 0),
    ([0x7FFFFFFF, 0x7FFFFFFF, 5], 3),
    ([0x40000000] * 4 + [3], 3),
    ([-1, 4], 3),
    ([5, 1], 3),
])
def test_inconsistent_group_sizes_are_flagged_without_out_of_range_reads(planner, gsz, ns):
    ng = len(gsz)
    cu_p = list(range(ng + 1))          # one prefix row per group: valid
    cu_s = list(range(ns + 1))          # one row per member: valid
    for mode in (0, 1):
        err, q, k, _ = run_plan(planner, cu_p, cu_s, gsz, ng, ns, ng, ns, mode=mode)
        assert err == 1 and not q and not k


@pytest.mark.parametrize("bad", ["cu_p_start", "cu_p_total", "cu_p_order", "cu_s_total", "cu_s_order", "size_sum"])
def test_inconsistent_offsets_are_flagged(planner, bad):
    cu_p, cu_s, gsz = (list(a) for a in arrays([5, 3], [2, 1], [4, 0, 6]))
    ng, ns, tp, ts = 2, 3, 8, 10
    if bad == "cu_p_start":
        cu_p[0] = 1
    elif bad == "cu_p_total":
        tp = 9
    elif bad == "cu_p_order":
        cu_p[1] = 9
    elif bad == "cu_s_total":
        ts = 11
    elif bad == "cu_s_order":
        cu_s[1] = 7
    else:
        gsz = [2, 2]
    for mode in (0, 1):
        err, q, k, _ = run_plan(planner, cu_p, cu_s, gsz, ng, ns, tp, ts, mode=mode)
        assert err == 1 and not q and not k


def expected_tiles(prefix, groups, suffix, kvc, split=0):
    """The tiling the kernels assume, as sets of (kind, group, row0, row1, aux, chunk, nchunks): prefix tiles
    of every group; response rows of a group stacked into tiles across member boundaries, or with ``split``
    each member's rows tiled on their own."""
    cu_p, cu_s, _ = arrays(prefix, groups, suffix)
    q, k = set(), set()
    m = 0
    for g, (p, gs) in enumerate(zip(prefix, groups)):
        p0, p1 = int(cu_p[g]), int(cu_p[g + 1])
        spans = ([(int(cu_s[i]), int(cu_s[i + 1])) for i in range(m, m + gs)] if split
                 else [(int(cu_s[m]), int(cu_s[m + gs]))])
        owner = lambda row: int(np.searchsorted(cu_s, row, side="right") - 1)  # noqa: E731
        for r0 in range(p0, p1, BM):
            q.add((0, g, r0, min(r0 + BM, p1), 0, 0, 1))
        for r0 in range(p0, p1, BKV):
            for c in range(kvc):
                k.add((0, g, r0, min(r0 + BKV, p1), 0, c, kvc))
        for s0, s1 in spans:
            for r0 in range(s0, s1, BM):
                q.add((1, g, r0, min(r0 + BM, s1), int(cu_s[owner(r0)]), 0, 1))
            for r0 in range(s0, s1, BKV):
                r1 = min(r0 + BKV, s1)
                k.add((1, g, r0, r1, int(cu_s[owner(r1 - 1) + 1]), 0, 1))
        m += gs
    return q, k


def check_loads(prefix, groups, suffix, q, k, seg, h_q, h_kv, d, dtype):
    """Every tensor row range the kernels load from a planned tile lies inside its tensor, and every
    buffer range (valid rows of one staged tile x row bytes) stays below 2^31 bytes."""
    cu_p, cu_s, _ = arrays(prefix, groups, suffix)
    tp, ts = int(cu_p[-1]), int(cu_s[-1])
    el = 2 if dtype == "bf16" else 4
    bq = BQ[dtype]
    gm = np.concatenate([[0], np.cumsum(groups)]).astype(np.int64)
    rng_pre = {g: (int(cu_p[g]), int(cu_p[g + 1])) for g in range(len(prefix))}
    rng_suf = {g: (int(cu_s[gm[g]]), int(cu_s[gm[g + 1]])) for g in range(len(prefix))}
    assert seg == cu_s[np.searchsorted(cu_s, np.arange(ts), side="right") - 1].tolist()

    def rows_ok(lo, hi, n, what):
        assert 0 <= lo < hi <= n, (what, lo, hi, n)

    for (kind, g, row0, row1, aux, work, chunk, nch) in q:
        p0, p1 = rng_pre[g]
        # the tile's own query rows (loaded row by row, clamped to row1 - 1)
        rows_ok(row0, row1, ts if kind else tp, "query rows")
        segs = [(p0, row1 if kind == 0 else p1, tp)] + ([(aux, row1, ts)] if kind else [])
        for lo, hi, n in segs:
            for k0 in range(lo, hi, BN):
                valid = min(BN, hi - k0)
                rows_ok(k0, k0 + valid, n, "key tile")
                assert valid * h_kv * d * el < 2 ** 31
        if kind:
            assert rng_suf[g][0] <= aux <= row0
    for (kind, g, row0, row1, aux, work, chunk, nch) in k:
        p0, p1 = rng_pre[g]
        s0, s1 = rng_suf[g]
        rows_ok(row0, row1, ts if kind else tp, "key rows")
        ranges = [(s0, s1, ts), (row0, p1, tp)] if kind == 0 else [(row0, aux, ts)]
        for lo, hi, n in ranges:
            for q0 in range(lo, hi, bq):
                valid = min(bq, hi - q0)
                rows_ok(q0, q0 + valid, n, "query tile")
                assert valid * h_q * d * el < 2 ** 31


def _planned(planner, prefix, groups, suffix, h_q, h_kv, modes=(0, 1), split=None):
    """Plans of the one-block planner (only where the library uses it: both tile lists within one block)
    and of the multi-kernel planner; modes=None: the planner the library would run. ``split`` defaults to
    the library's choice."""
    cu_p, cu_s, gsz = arrays(prefix, groups, suffix)
    ng, ns, tp, ts = len(prefix), len(suffix), int(cu_p[-1]), int(cu_s[-1])
    kvc = kv_chunks_for(ng, tp, ts, h_q, h_kv)
    split = split_for(ng, tp, ts, h_q) if split is None else split
    max_q, max_kv = bounds(ng, ns, tp, ts, kvc)
    one_block = max_q <= 1024 and max_kv <= 1024
    if modes is None:
        modes = (0,) if one_block else (1,)
    plans = [run_plan(planner, cu_p, cu_s, gsz, ng, ns, tp, ts, mode=mode, kvc=kvc, split=split)
             for mode in modes if mode == 1 or one_block]
    return plans, kvc, split


@pytest.mark.parametrize("seed,split", [(s, s % 2) for s in range(6)])
def test_random_groupings_plan_as_the_kernels_assume(planner, seed, split):
    rng = np.random.default_rng(seed)
    ng = int(rng.integers(1, 40))
    prefix = rng.integers(0, 600, ng) * (rng.random(ng) < 0.8)
    groups = rng.integers(0, 6, ng)
    suffix = rng.integers(0, 400, int(groups.sum())) * (rng.random(int(groups.sum())) < 0.9)
    (fused, multi), kvc, _ = _planned(planner, prefix, groups, suffix, 8, 2, split=split)
    assert fused == multi
    err, q, k, seg = fused
    assert err == 0
    eq, ek = expected_tiles(list(prefix), list(groups), list(suffix), kvc, split)
    assert set(t[:5] + t[6:] for t in q) == eq and len(q) == len(eq)
    assert set(t[:5] + t[6:] for t in k) == ek and len(k) == len(ek)
    for tiles in (q, k):
        work = [t[5] for t in tiles]
        assert work == sorted(work, reverse=True)
    check_loads(prefix, groups, suffix, q, k, seg, 8, 2, 128, "bf16")


@pytest.mark.parametrize("name", ["tiny", "single_group", "long_prefix", "large_group", "packed_varlen"])
def test_workload_loads_stay_in_range(planner, name):
    wl = WORKLOADS[name]
    prefix, groups, suffix = draw_lengths(wl, 0)
    plans, _, _ = _planned(planner, prefix, groups, suffix, wl.h_q, wl.h_kv)
    assert all(p == plans[0] for p in plans) and plans[0][0] == 0
    _, q, k, seg = plans[0]
    check_loads(prefix, groups, suffix, q, k, seg, wl.h_q, wl.h_kv, wl.head_dim, wl.dtype)


def test_fig23_grid_loads_stay_in_range(planner):
    """Corners of the bench sweep's grid (P 4096/16384, G 2/16, responses around P/r for r = 1, 16; the
    middle points plan the same way), plus the 2 GiB dense query range that once overran its buffer
    (16 members of 1024 rows at h_q * d = 65536)."""
    for P in (4096, 16384):
        for G in (2, 16):
            for r in (1, 16):
                S = P // r
                wl = Workload("grid", 1, G, ("fixed", P), ("uniform", S // 2, S + S // 2), 32, 8, 128, "bf16", 1.0)
                prefix, groups, suffix = draw_lengths(wl, 0)
                (plan,), _, _ = _planned(planner, prefix, groups, suffix, 32, 8, modes=None)
                check_loads(prefix, groups, suffix, plan[1], plan[2], plan[3], 32, 8, 128, "bf16")
    prefix, groups, suffix = [128], [16], [1024] * 16
    (plan,), _, _ = _planned(planner, prefix, groups, suffix, 512, 64, modes=None)
    check_loads(prefix, groups, suffix, plan[1], plan[2], plan[3], 512, 64, 128, "bf16")

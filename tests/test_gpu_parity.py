"""GPU parity: the HIP library against the CPU oracle on the same seeded inputs.

Small problems are compared element by element on every output and gradient;
the five workloads are compared at full size in the launch configuration the
bench uses, either on every element of a subset of heads (single_group) or on
sampled query rows and keys the oracle computes one by one.
"""
import os

import numpy as np
import pytest

from oracle import grouped_oracle, key_gradients, query_rows
from paper_2506_05433_amd.inputs import make_problem
from tests._parity import GRADS, OUTS, check, host_view, to_host

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _dev():
    from paper_2506_05433_amd import binding
    assert torch.cuda.is_available(), "GPU test needs a GPU"
    binding.lib()
    return binding


def _run(prob, grads=True):
    binding = _dev()
    dev = binding.to_device(prob, "cuda")
    f = binding.run_fwd(dev)
    res = dict(zip(OUTS, f))
    if grads:
        res.update(zip(GRADS, binding.run_bwd(dev, f)))
    torch.cuda.synchronize()
    return {k: to_host(v) for k, v in res.items()}


def _oracle(prob, grads, heads):
    """Full oracle; with ``heads``, one thread per query head (numpy releases the GIL), results merged."""
    t = host_view(prob)
    args = (prob.prefix_lens, prob.group_sizes, prob.suffix_lens)
    if heads is None:
        return grouped_oracle(*args, t, prob.scale, grads=grads)
    from concurrent.futures import ThreadPoolExecutor
    tf = {k: np.asarray(v, np.float64) for k, v in t.items()}
    with ThreadPoolExecutor(len(heads)) as ex:
        parts = list(ex.map(lambda h: grouped_oracle(*args, tf, prob.scale, grads=grads, heads=[h]), heads))
    ref = {k: (sum(p[k] for p in parts) if k in ("dk_pre", "dk_suf", "dv_pre", "dv_suf", "prefix_member_spread")
               else None) for k in parts[0]}
    for k in parts[0]:
        if ref[k] is None:
            ref[k] = parts[0][k].copy()
            for h, p in zip(heads, parts):
                if k.startswith("lse"):
                    ref[k][h] = p[k][h]
                else:
                    ref[k][:, h] = p[k][:, h]
    return ref


def _full_compare(prob, grads=True, heads=None, kv_heads=None):
    print(f"[parity] {prob.workload.name} seed={prob.seed} P={list(prob.prefix_lens)} G={list(prob.group_sizes)} "
          f"S={list(prob.suffix_lens)[:8]}... hq={prob.h_q} hkv={prob.h_kv} d={prob.head_dim} {prob.dtype}",
          flush=True)
    got = _run(prob, grads)
    ref = _oracle(prob, grads, heads)
    assert ref["prefix_member_spread"] == 0.0
    hs = slice(None) if heads is None else list(heads)
    for k in OUTS:
        if k.startswith("lse"):
            check(k, got[k][hs], ref[k][hs], prob.dtype)
        else:
            check(k, got[k][:, hs], ref[k][:, hs], prob.dtype)
    if grads:
        ks = slice(None) if kv_heads is None else list(kv_heads)
        for k in GRADS:
            sel = hs if k.startswith("dq") else ks
            check(k, got[k][:, sel], ref[k][:, sel], prob.dtype)
    return got


def test_tiny_fp32_workload():
    """The 'tiny' workload (fp32, d=64) element by element."""
    _full_compare(make_problem("tiny", seed=0))


SMALL = [
    # (lengths, h_q, h_kv, d, dtype): several tiles, ragged tails, GQA ratios 1/4/5/8, edge sizes
    (((300,), (5,), (130, 1, 64, 200, 97)), 8, 2, 128, "bf16"),
    (((257, 0, 40), (3, 2, 0), (129, 128, 1, 300, 0)), 5, 1, 128, "bf16"),
    (((1000,), (4,), (70, 250, 33, 190)), 8, 1, 128, "bf16"),
    (((190,), (3,), (64, 65, 127)), 4, 4, 64, "bf16"),
    (((513, 77), (2, 3), (200, 5, 64, 1, 300)), 4, 2, 64, "bf16"),
    (((300,), (5,), (130, 1, 64, 200, 97)), 4, 2, 128, "fp32"),
    (((129, 0), (2, 2), (40, 63, 1, 128)), 2, 1, 64, "fp32"),
    (((0,), (1,), (5,)), 2, 2, 64, "bf16"),
    (((7,), (0,), ()), 2, 1, 128, "bf16"),
    # many groups: empty groups, a group without prefix, prefixes shorter than a tile, GQA ratio 8
    (((3, 0, 200, 1), (2, 1, 0, 3), (5, 0, 7, 1, 1, 130)), 8, 1, 128, "bf16"),
    # GQA ratio 5 with head_dim 64
    (((150,), (2,), (77, 200)), 5, 1, 64, "bf16"),
    # the head geometries of the full-size workloads (8 kv heads: the XCD head-mapping branch that gives
    # each XCD one kv head), every element of every head
    (((300,), (3,), (130, 64, 200)), 32, 8, 128, "bf16"),
    (((257,), (3,), (100, 1, 190)), 40, 8, 128, "bf16"),
    (((200, 130), (2, 2), (70, 129, 5, 60)), 64, 8, 128, "bf16"),
]


@pytest.mark.parametrize("case", range(len(SMALL)))
def test_small_full(case):
    lengths, hq, hkv, d, dt = SMALL[case]
    prob = make_problem("single_group", seed=100 + case, lengths=lengths, h_q=hq, h_kv=hkv, head_dim=d, dtype=dt,
                        scale=1.0 / np.sqrt(d))
    _full_compare(prob)


def test_more_groups_than_one_planner_pass():
    """1100 groups, more than the planner's 1024 threads scan in one pass (and the multi-kernel planner,
    since the tile lists no longer fit one block): tiny prefixes and responses, empty ones included,
    every output and gradient against the oracle."""
    rng = np.random.default_rng(11)
    ng = 1100
    prefix = rng.integers(0, 6, ng)
    groups = rng.integers(0, 3, ng)
    suffix = rng.integers(0, 5, int(groups.sum()))
    prob = make_problem("single_group", seed=11, lengths=(prefix, groups, suffix), h_q=2, h_kv=1, head_dim=64,
                        dtype="fp32", scale=0.125)
    print(f"[parity] {ng} groups, {len(suffix)} members, total_prefix={prob.total_prefix} "
          f"total_suffix={prob.total_suffix}", flush=True)
    _full_compare(prob)


def test_peaked_softmax_rescaling():
    """Q x 4: sharp rows exercise the running-max rescale of the online softmax."""
    prob = make_problem("single_group", seed=7, lengths=((700,), (3,), (300, 90, 211)), h_q=4, h_kv=1,
                        head_dim=128, peaked=True)
    _full_compare(prob)


def test_single_group_workload_every_head():
    """single_group (P=4096, G=8, 32/8 heads) at full size: every element of every head."""
    prob = make_problem("single_group", seed=0)
    _full_compare(prob, heads=list(range(prob.h_q)))


def _tiles(lo, hi, bm=128):
    """(first row, last row) of every bm-row tile of [lo, hi) (the planner's query tiles)."""
    return [(a, min(a + bm, hi) - 1) for a in range(lo, hi, bm)]


def _identities(prob, got_dev, dev):
    """Over every group and kv head, on the GPU's own results: sum of dV over the group's keys = sum of dO
    over the group's queries and the kv head's query heads (softmax rows sum to one), and sum of dK = 0
    (every row of dS sums to zero), relative to sum |dK|."""
    ratio = prob.h_q // prob.h_kv
    cu_p, cu_s = prob.cu_prefix, prob.cu_suffix
    m = 0
    worst_v = worst_k = 0.0
    for g, gs in enumerate(prob.group_sizes):
        p0, p1 = int(cu_p[g]), int(cu_p[g + 1])
        s0, s1 = int(cu_s[m]), int(cu_s[m + int(gs)])
        m += int(gs)
        if p1 == p0 and s1 == s0:
            continue

        def seg(t, a, b):
            return t[a:b].double().sum(0)

        dv = seg(got_dev["dv_pre"], p0, p1) + seg(got_dev["dv_suf"], s0, s1)            # [h_kv, d]
        do = seg(dev["do_pre"], p0, p1) + seg(dev["do_suf"], s0, s1)                    # [h_q, d]
        do = do.view(prob.h_kv, ratio, -1).sum(1)
        dk = seg(got_dev["dk_pre"], p0, p1) + seg(got_dev["dk_suf"], s0, s1)
        dk_abs = got_dev["dk_pre"][p0:p1].double().abs().sum(0) + got_dev["dk_suf"][s0:s1].double().abs().sum(0)
        rv = float(((dv - do).abs().amax(1) / do.abs().amax(1).clamp_min(1e-30)).max())
        assert bool((dk_abs.amax(1) > 0).all()), f"group {g}: a kv head has all-zero dK"
        rk = float((dk.abs().amax(1) / dk_abs.amax(1)).max())
        worst_v, worst_k = max(worst_v, rv), max(worst_k, rk)
    print(f"identities over {len(prob.group_sizes)} groups x {prob.h_kv} kv heads: "
          f"sum dV vs sum dO rel={worst_v:.3e}; |sum dK| / sum |dK| = {worst_k:.3e}", flush=True)
    assert worst_v < 3e-2 and worst_k < 1e-2


def _sampled_compare(prob, head_groups=1, kv_group=0, kv_heads=None, n_keys=4, seed=0):
    """Full-size workload against the oracle on sampled outputs, float32 oracle.

    * query side: the first and last row of every query tile (prefix tiles of every group, response
      tiles stacked over the members of every group), every query head (with ``head_groups`` > 1, tile i
      takes the heads h with h % head_groups == i % head_groups, so every head and every tile is covered);
      O, LSE and dQ;
    * key side: dK, dV of keys of group ``kv_group`` for every kv head in ``kv_heads`` (default all):
      the last prefix keys (where the causal prefix rows end), a few random prefix keys near the end, the
      first and last response keys of the first and last member, and random response keys;
    * the sum identities over every group and kv head.
    """
    print(f"[parity] sampled {prob.workload.name} seed={prob.seed} total_prefix={prob.total_prefix} "
          f"total_suffix={prob.total_suffix}", flush=True)
    binding = _dev()
    dev = binding.to_device(prob, "cuda")
    f = binding.run_fwd(dev)
    g = binding.run_bwd(dev, f)
    torch.cuda.synchronize()
    got_dev = dict(zip(OUTS, f))
    got_dev.update(zip(GRADS, g))
    _identities(prob, got_dev, dev)
    t = host_view(prob)
    rng = np.random.default_rng(seed)
    hq = prob.h_q
    cu_p, cu_s = prob.cu_prefix, prob.cu_suffix
    args = (prob.prefix_lens, prob.group_sizes, prob.suffix_lens, t, prob.scale)
    m = 0
    pre_tiles, suf_tiles = [], []
    for gi, gs in enumerate(prob.group_sizes):
        pre_tiles += _tiles(int(cu_p[gi]), int(cu_p[gi + 1]))
        suf_tiles += _tiles(int(cu_s[m]), int(cu_s[m + int(gs)]))
        m += int(gs)
    for side, tiles in (("pre", pre_tiles), ("suf", suf_tiles)):
        for hg in range(head_groups):
            heads = [h for h in range(hq) if h % head_groups == hg]
            rows = sorted(set(r for i, tr in enumerate(tiles) if i % head_groups == hg for r in tr))
            if not rows:
                continue
            r = query_rows(*args, side, rows, heads, dtype=np.float32)
            idx_r = torch.tensor(rows, device="cuda")
            idx_h = torch.tensor(heads, device="cuda")
            check("o_" + side, to_host(got_dev["o_" + side][idx_r][:, idx_h]), r["o"], prob.dtype)
            check("lse_" + side, to_host(got_dev["lse_" + side][idx_h][:, idx_r]), r["lse"], prob.dtype)
            check("dq_" + side, to_host(got_dev["dq_" + side][idx_r][:, idx_h]), r["dq"], prob.dtype)
    gq = kv_group
    p0, p1 = int(cu_p[gq]), int(cu_p[gq + 1])
    m0 = int(prob.group_sizes[:gq].sum())
    m1 = m0 + int(prob.group_sizes[gq])
    tail = max(p0, p1 - 300)
    pkeys = sorted(set([p1 - 1, p1 - 2, max(p0, p1 - 129)] + list(rng.integers(tail, p1, n_keys))))
    skeys = sorted(set([int(cu_s[m0]), int(cu_s[m0 + 1]) - 1, int(cu_s[m1 - 1]), int(cu_s[m1]) - 1] +
                       list(rng.integers(cu_s[m0], cu_s[m1], n_keys))))
    for kv in (range(prob.h_kv) if kv_heads is None else kv_heads):
        for side, keys in (("pre", pkeys), ("suf", skeys)):
            r = key_gradients(*args, gq, kv, side, keys, dtype=np.float32)
            idx = torch.tensor(keys, device="cuda")
            check(f"dk_{side}[kv{kv}]", to_host(got_dev["dk_" + side][idx, kv]), r["dk"], prob.dtype)
            check(f"dv_{side}[kv{kv}]", to_host(got_dev["dv_" + side][idx, kv]), r["dv"], prob.dtype)


def test_long_prefix_workload_sampled():
    """long_prefix (P=16384, G=16, 32/8): every tile, every head; dK/dV of every kv head."""
    _sampled_compare(make_problem("long_prefix", seed=0))


def test_large_group_workload_sampled():
    """large_group (P=8192, G=64, 40/8): every tile, every head; dK/dV of kv heads 0 and 7."""
    _sampled_compare(make_problem("large_group", seed=0), kv_heads=[0, 7])


def test_packed_varlen_workload_sampled():
    """packed_varlen (8 groups, 64/8): every tile with 8 of its heads (every head over eight tiles in
    turn); dK/dV of every kv head of the group with the shortest prefix."""
    prob = make_problem("packed_varlen", seed=0)
    _sampled_compare(prob, head_groups=8, kv_group=int(np.argmin(prob.prefix_lens)))


def test_deterministic():
    """Two runs on identical inputs are bitwise equal (fixed-order reductions, no atomics)."""
    prob = make_problem("single_group", seed=3, lengths=((900,), (6,), (100, 300, 1, 250, 64, 129)), h_q=8, h_kv=2,
                        head_dim=128)
    a = _run(prob)
    b = _run(prob)
    for k in a:
        assert np.array_equal(a[k], b[k]), k


def test_repeated_layout_sums_to_grouped():
    """The same kernels on the repeated-prefix layout give the grouped results (Lemma 1 on the GPU)."""
    from paper_2506_05433_amd.inputs import repeated_layout
    prob = make_problem("single_group", seed=4, lengths=((520,), (3,), (100, 7, 260)), h_q=4, h_kv=1, head_dim=128,
                        dtype="fp32")
    rep = repeated_layout(prob)
    g = _run(prob)
    r = _run(rep)
    P = int(prob.prefix_lens[0])
    np.testing.assert_allclose(r["o_suf"], g["o_suf"], atol=1e-5)
    for i in range(3):
        np.testing.assert_allclose(r["o_pre"][i * P:(i + 1) * P], g["o_pre"], atol=1e-5)
    for name in ("dk_pre", "dv_pre", "dq_pre"):
        s = sum(r[name][i * P:(i + 1) * P] for i in range(3))
        np.testing.assert_allclose(s, g[name], atol=1e-4)


def test_invalid_grouping_arrays_do_no_work(monkeypatch):
    """Inconsistent device grouping arrays: nothing is computed, and PG_DEBUG_VALIDATE=1 reports PG_EINVAL."""
    binding = _dev()
    prob = make_problem("single_group", seed=5, lengths=((64,), (2,), (10, 20)), h_q=2, h_kv=1, head_dim=64)
    dev = binding.to_device(prob, "cuda")
    dev["cu_suffix"] = torch.tensor([0, 25, 20], dtype=torch.int32, device="cuda")  # not nondecreasing
    o_pre = torch.full_like(dev["q_pre"], 7.0)
    o_suf = torch.full_like(dev["q_suf"], 7.0)
    lp = torch.zeros(2, 64, device="cuda")
    ls = torch.zeros(2, 30, device="cuda")
    binding.fwd(dev["q_pre"], dev["k_pre"], dev["v_pre"], dev["q_suf"], dev["k_suf"], dev["v_suf"],
                dev["cu_prefix"], dev["cu_suffix"], dev["group_sizes"], dev["scale"], out=(o_pre, o_suf, lp, ls))
    torch.cuda.synchronize()
    assert bool((o_pre == 7.0).all()) and bool((o_suf == 7.0).all())
    # the device's verdict, read back from the call's workspace on request
    ws = torch.empty(binding.workspace_bytes("fwd", 1, 2, 64, 30, 2, 1, 64), device="cuda", dtype=torch.uint8)
    binding.fwd(dev["q_pre"], dev["k_pre"], dev["v_pre"], dev["q_suf"], dev["k_suf"], dev["v_suf"],
                dev["cu_prefix"], dev["cu_suffix"], dev["group_sizes"], dev["scale"], out=(o_pre, o_suf, lp, ls),
                workspace=ws)
    with pytest.raises(binding.PgError) as e:
        binding.plan_status(ws)
    assert e.value.status == 1
    good = binding.to_device(prob, "cuda")
    binding.fwd(good["q_pre"], good["k_pre"], good["v_pre"], good["q_suf"], good["k_suf"], good["v_suf"],
                good["cu_prefix"], good["cu_suffix"], good["group_sizes"], good["scale"], workspace=ws)
    binding.plan_status(ws)
    monkeypatch.setenv("PG_DEBUG_VALIDATE", "1")
    with pytest.raises(binding.PgError) as e:
        binding.fwd(dev["q_pre"], dev["k_pre"], dev["v_pre"], dev["q_suf"], dev["k_suf"], dev["v_suf"],
                    dev["cu_prefix"], dev["cu_suffix"], dev["group_sizes"], dev["scale"])
    assert e.value.status == 1


def test_dense_query_range_of_two_gib():
    """A prefix key tile whose dense query range (every response row of the group) spans 2^31 bytes.

    16 members of 1024 rows and h_q * head_dim = 65536 give 16384 rows of 128 KiB: the byte range
    of the staged query tiles must be that of the tile, not of the whole remaining range. Checked on
    sampled rows and keys against the oracle, and on sum dV = sum dO and sum dK = 0 over every key
    of kv head 0 (the softmax rows sum to one; each row of dS sums to zero).
    """
    prob = make_problem("single_group", seed=3, lengths=([128], [16], [1024] * 16), h_q=512, h_kv=64)
    print(f"[parity] dense 2 GiB range: total_prefix={prob.total_prefix} total_suffix={prob.total_suffix} "
          f"h_q={prob.h_q} h_kv={prob.h_kv}", flush=True)
    binding = _dev()
    dev = binding.to_device(prob, "cuda")
    f = binding.run_fwd(dev)
    g = binding.run_bwd(dev, f)
    torch.cuda.synchronize()
    out = dict(zip(OUTS, f))
    out.update(zip(GRADS, g))
    t = host_view(prob)
    heads = [0, 7, 300, 511]
    rows = [0, 1023, 1024, 8191, 16383]
    r = query_rows(prob.prefix_lens, prob.group_sizes, prob.suffix_lens, t, prob.scale, "suf", rows, heads)
    idx_r, idx_h = torch.tensor(rows, device="cuda"), torch.tensor(heads, device="cuda")
    check("o_suf", to_host(out["o_suf"][idx_r][:, idx_h]), r["o"], prob.dtype)
    check("dq_suf", to_host(out["dq_suf"][idx_r][:, idx_h]), r["dq"], prob.dtype)
    keys = [0, 64, 127]
    r = key_gradients(prob.prefix_lens, prob.group_sizes, prob.suffix_lens, t, prob.scale, 0, 0, "pre", keys)
    check("dk_pre", to_host(out["dk_pre"][keys, 0]), r["dk"], prob.dtype)
    check("dv_pre", to_host(out["dv_pre"][keys, 0]), r["dv"], prob.dtype)
    ratio = prob.h_q // prob.h_kv
    dv_sum = out["dv_pre"][:, 0].double().sum(0) + out["dv_suf"][:, 0].double().sum(0)
    do_sum = dev["do_pre"][:, :ratio].double().sum((0, 1)) + dev["do_suf"][:, :ratio].double().sum((0, 1))
    rel = float((dv_sum - do_sum).abs().max() / do_sum.abs().max())
    dk = torch.cat([out["dk_pre"][:, 0], out["dk_suf"][:, 0]]).double()
    rel_k = float(dk.sum(0).abs().max() / dk.abs().sum(0).max())
    print(f"sum dV vs sum dO rel={rel:.3e}; |sum dK| / sum |dK| = {rel_k:.3e}", flush=True)
    assert rel < 3e-2 and rel_k < 1e-2

"""Host-side checks of bench.py (no GPU): the useful-pair count, the one-GPU contract and the
counter bookkeeping."""
import json
import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def brute_pairs(prefix_lens, group_sizes, suffix_lens):
    """Count allowed (query, key) pairs by enumerating the visibility rule of Eq. (4)."""
    total, m = 0, 0
    for p, g in zip(prefix_lens, group_sizes):
        total += sum(1 for t in range(p) for s in range(p) if s <= t)
        for s_len in suffix_lens[m:m + g]:
            total += sum(1 for j in range(s_len) for s in range(p + s_len) if s < p or s - p <= j)
        m += g
    return total


def test_pair_count_matches_enumeration():
    rng = np.random.default_rng(0)
    for _ in range(20):
        ng = int(rng.integers(1, 4))
        prefix = rng.integers(0, 12, ng)
        groups = rng.integers(0, 4, ng)
        suffix = rng.integers(0, 9, int(groups.sum()))
        assert bench.pair_count(prefix, groups, suffix) == brute_pairs(prefix, groups, suffix)


def test_repeated_pairs_and_eq17_limit():
    # Appendix A.2, Eq. (15)-(18): with equal response lengths the ratio of repeated to grouped pairs
    # tends to G as the prefix grows
    G, Lr = 8, 4
    for Lp, lo in ((10, 1.0), (1000, 7.0), (100000, 7.99)):
        r = bench.repeated_pair_count([Lp], [G], [Lr] * G) / bench.pair_count([Lp], [G], [Lr] * G)
        assert lo <= r <= G


def test_more_than_one_gpu_is_refused():
    out = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                         text=True)
    assert out.returncode == 2 and "one GPU" in out.stderr


def test_traffic_is_reported_only_for_the_profiled_sources(tmp_path, monkeypatch):
    import shutil
    shutil.copytree(os.path.join(bench.ROOT, "paper_2506_05433_amd", "csrc"),
                    tmp_path / "paper_2506_05433_amd" / "csrc")
    prof = tmp_path / "profiles"
    prof.mkdir()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    rec = dict(kernel="dkdv", workload="w", source_sha="not-this-build", copy_read_bytes=1 << 30,
               copy_write_bytes=1 << 30, copy_fetch_kib=524288.0, copy_write_kib=1048576.0, fetch_kib=1000.0,
               write_kib=10.0)
    (prof / "traffic_dkdv_w.json").write_text(json.dumps(rec))
    assert bench.recorded_traffic("dkdv", "w") is None
    digest = bench.kernel_source_sha()
    rec["source_sha"] = digest
    (prof / "traffic_dkdv_w.json").write_text(json.dumps(rec))
    assert bench.recorded_traffic("dkdv", "w") == 1000.0 * 1024 * 2 + 10.0 * 1024 * 1
    # sources the attention kernels are not built from do not invalidate the reading ...
    with open(tmp_path / "paper_2506_05433_amd" / "csrc" / "pg_rope.hpp", "a") as fh:
        fh.write("// edit\n")
    assert bench.kernel_source_sha() == digest
    # ... an edit of theirs does
    with open(tmp_path / "paper_2506_05433_amd" / "csrc" / "pg_bwd.hpp", "a") as fh:
        fh.write("// edit\n")
    assert bench.kernel_source_sha() != digest
    assert bench.recorded_traffic("dkdv", "w") is None


def _cpu_dev(prob):
    import torch
    out = {}
    for name, a in prob.tensors.items():
        t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16) if a.dtype == np.uint16 \
            else torch.from_numpy(np.ascontiguousarray(a))
        out[name] = t
    out["scale"] = prob.scale
    return out


def test_device_repeated_layout_matches_host_construction():
    """bench's repeated layout (built with index_select) equals inputs.repeated_layout, empty groups included."""
    from paper_2506_05433_amd.inputs import make_problem, repeated_layout
    import torch
    prob = make_problem("single_group", seed=2, lengths=((5, 0, 7, 3), (2, 1, 0, 3), (4, 0, 6, 1, 2, 3)), h_q=4,
                        h_kv=2, head_dim=64)
    got, shape = bench.baseline_layout(torch, _cpu_dev(prob), prob, padded=False)
    ref = repeated_layout(prob)
    assert shape == bench.shape_of(ref)
    assert got["cu_prefix"].tolist() == ref.cu_prefix.tolist()
    assert got["cu_suffix"].tolist() == ref.cu_suffix.tolist()
    assert got["group_sizes"].tolist() == ref.group_sizes.tolist()
    for name, a in ref.tensors.items():
        assert np.array_equal(got[name].view(torch.int16).numpy().view(np.uint16), a), name


def test_device_padded_layout():
    """Padded layout of Eq. (1): member i of a group keeps its rows and gets zero rows up to the group's
    longest response; pair count = sum over members of (P + max S)(P + max S + 1) / 2."""
    from paper_2506_05433_amd.inputs import make_problem
    import torch
    lengths = ((5, 3), (3, 2), (4, 1, 6, 2, 2))
    prob = make_problem("single_group", seed=2, lengths=lengths, h_q=2, h_kv=1, head_dim=64, dtype="fp32")
    got, shape = bench.baseline_layout(torch, _cpu_dev(prob), prob, padded=True)
    assert got["cu_suffix"].tolist() == [0, 6, 12, 18, 20, 22]
    assert got["cu_prefix"].tolist() == [0, 5, 10, 15, 18, 21]
    q = got["q_suf"].numpy()
    src = prob.tensors["q_suf"]
    assert np.array_equal(q[0:4], src[0:4]) and not q[4:6].any()
    assert np.array_equal(q[6:7], src[4:5]) and not q[7:12].any()
    assert np.array_equal(q[12:18], src[5:11])
    assert np.array_equal(q[20:22], src[13:15])
    # do_pre only on the first copy of each group's prefix
    dp = got["do_pre"].numpy()
    assert np.array_equal(dp[0:5], prob.tensors["do_pre"][0:5]) and not dp[5:15].any()
    assert bench.padded_pair_count(*lengths) == 3 * (11 * 12 // 2) + 2 * (5 * 6 // 2)
    assert bench.padded_pair_count(*lengths) == bench.repeated_pair_count(
        got["cu_prefix"].diff().numpy(), np.ones(5, int), got["cu_suffix"].diff().numpy())


def test_cpu_baseline_units_are_the_oracle_on_one_group_and_head():
    """The CPU leg's (group, head) sub-problem gives the full oracle's rows of that group and head."""
    from oracle import grouped_oracle
    from paper_2506_05433_amd.inputs import make_problem
    prob = make_problem("single_group", seed=3, lengths=((6, 4), (2, 3), (3, 1, 5, 2, 4)), h_q=4, h_kv=2,
                        head_dim=64)
    t = {k: prob.as_float(k) for k in prob.tensors}
    full = grouped_oracle(prob.prefix_lens, prob.group_sizes, prob.suffix_lens, t, prob.scale)
    lengths, sub = bench.sub_problem(prob, 1, 3)
    r = grouped_oracle(*lengths, sub, prob.scale)
    assert np.array_equal(r["o_pre"][:, 0], full["o_pre"][6:10, 3])
    assert np.array_equal(r["dq_suf"][:, 0], full["dq_suf"][4:15, 3])
    res = bench.cpu_baseline(prob, 1.0)
    assert res["kind"] == "oracle" and res["value"] > 0 and res["cores"] >= 1


def test_prefix_copy_sum_adds_each_groups_copies():
    """The repeated layout's separately timed extra step: the G-way sum of each group's prefix gradient copies,
    checked against a loop over the copies (groups of size 0 and 1 have nothing to add)."""
    from paper_2506_05433_amd.inputs import make_problem
    import torch
    prob = make_problem("single_group", seed=3, lengths=((5, 0, 7, 3), (2, 1, 0, 3), (4, 0, 6, 1, 2, 3)), h_q=4,
                        h_kv=2, head_dim=64)
    _, shape = bench.baseline_layout(torch, _cpu_dev(prob), prob, padded=False)
    rows = shape[2]
    g = torch.Generator().manual_seed(0)
    grads = tuple(torch.randn((rows, h, 64), generator=g) for h in (4, 2, 2))
    run = bench.copy_sum_fn(torch, prob, {"bwd": grads})
    run()
    # expected: walk the layout's prefix rows group by group
    row, k = 0, 0
    for p, gs in zip(prob.prefix_lens, prob.group_sizes):
        p, gs = int(p), int(gs)
        if gs > 1 and p > 0:
            for t, outs in zip(grads, run.outs):
                want = sum(t[row + i * p: row + (i + 1) * p] for i in range(gs))
                assert torch.allclose(outs[k], want, atol=1e-5)
            k += 1
        row += max(gs, 1) * p
    assert row == rows and k == len(run.outs[0]) == 2


def test_single_buffer_row_order():
    """inputs.xours_order: a permutation of the packed rows that puts, group after group, the prefix rows and
    then the group's members' response rows (Eq. (2)); empty groups and members included."""
    from paper_2506_05433_amd.inputs import make_problem, xours_order
    prob = make_problem("single_group", seed=2, lengths=((5, 0, 7, 3), (2, 1, 0, 3), (4, 0, 6, 1, 2, 3)), h_q=4,
                        h_kv=2, head_dim=64)
    order = xours_order(prob)
    tp = prob.total_prefix
    assert sorted(order.tolist()) == list(range(tp + prob.total_suffix))
    row, m = 0, 0
    for g, gs in enumerate(prob.group_sizes):
        p0, p1 = int(prob.cu_prefix[g]), int(prob.cu_prefix[g + 1])
        s0, s1 = int(prob.cu_suffix[m]), int(prob.cu_suffix[m + int(gs)])
        assert order[row:row + p1 - p0].tolist() == list(range(p0, p1))
        row += p1 - p0
        assert order[row:row + s1 - s0].tolist() == [tp + r for r in range(s0, s1)]
        row += s1 - s0
        m += int(gs)
    assert row == len(order)

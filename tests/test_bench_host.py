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

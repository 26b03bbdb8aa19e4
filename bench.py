"""Benchmark: grouped (shared-prefix) attention forward+backward on one MI355X.

python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline] [--no-repeated]

A step is one forward and one backward call over the whole workload (inputs
resident in HBM). Prints ONE JSON line. ``value`` is useful TFLOP/s:
4*d*H_q*pairs (forward) + 10*d*H_q*pairs (backward) per step, where pairs is
the exact number of (query, key) pairs the grouped problem allows; masked
work, ragged tiles and the repeated-prefix pairs the method avoids are not
counted. The timed step is the forward and backward calls captured once as a
HIP graph and replayed (the eager time of the same calls is reported too;
per-kernel times come from HIP events in the eager pass). The same kernels
are also timed on the repeated-prefix layout (every member with its own copy
of the prefix) for the speedup.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "grouped attn fwd+bwd TFLOP/s (useful) & % MFMA peak; speedup vs repeated-prefix"
PEAK_TFLOPS = {"bf16": 2500.0, "fp32": 157.3}


def pair_count(prefix_lens, group_sizes, suffix_lens):
    """Allowed (query, key) pairs of the grouped problem: prefix row t sees t+1 keys, response row j sees P+j+1."""
    total = 0
    m = 0
    for p, g in zip(prefix_lens, group_sizes):
        p = int(p)
        total += p * (p + 1) // 2
        for s in suffix_lens[m:m + int(g)]:
            s = int(s)
            total += s * p + s * (s + 1) // 2
        m += int(g)
    return total


def repeated_pair_count(prefix_lens, group_sizes, suffix_lens):
    total, m = 0, 0
    for p, g in zip(prefix_lens, group_sizes):
        for s in suffix_lens[m:m + int(g)]:
            n = int(p) + int(s)
            total += n * (n + 1) // 2
        m += int(g)
    return total


def progress(msg):
    """A progress line on stderr (the JSON result is the only stdout line)."""
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def time_steps(binding, torch, dev, bufs, steps, warmup):
    def step():
        binding.fwd(dev["q_pre"], dev["k_pre"], dev["v_pre"], dev["q_suf"], dev["k_suf"], dev["v_suf"],
                    dev["cu_prefix"], dev["cu_suffix"], dev["group_sizes"], dev["scale"], out=bufs["fwd"],
                    workspace=bufs["ws_f"])
        o_pre, o_suf, lse_pre, lse_suf = bufs["fwd"]
        binding.bwd(dev["q_pre"], dev["k_pre"], dev["v_pre"], dev["q_suf"], dev["k_suf"], dev["v_suf"],
                    o_pre, o_suf, lse_pre, lse_suf, dev["do_pre"], dev["do_suf"],
                    dev["cu_prefix"], dev["cu_suffix"], dev["group_sizes"], dev["scale"], out=bufs["bwd"],
                    workspace=bufs["ws_b"])

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    binding.timing_start()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    binding.timing_stop()
    ms = e0.elapsed_time(e1) / steps
    kern = {}
    for k in ("plan", "fwd", "dkdv", "dq"):
        n, tot = binding.timing_get(k)
        kern[k] = {"launches": n, "avg_ms": (tot / n) if n else None}
    # the same step captured once as a HIP graph and replayed: no host launch cost per kernel
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    for _ in range(warmup):
        graph.replay()
    torch.cuda.synchronize()
    e0.record()
    for _ in range(steps):
        graph.replay()
    e1.record()
    torch.cuda.synchronize()
    ms_graph = e0.elapsed_time(e1) / steps
    del graph
    return ms_graph, kern, ms


def alloc(binding, torch, dev, prob):
    bufs = {
        "fwd": (torch.empty_like(dev["q_pre"]), torch.empty_like(dev["q_suf"]),
                torch.empty((prob.h_q, prob.total_prefix), device="cuda", dtype=torch.float32),
                torch.empty((prob.h_q, prob.total_suffix), device="cuda", dtype=torch.float32)),
        "bwd": tuple(torch.empty_like(dev[k]) for k in ("q_pre", "k_pre", "v_pre", "q_suf", "k_suf", "v_suf")),
    }
    args = (len(prob.prefix_lens), len(prob.suffix_lens), prob.total_prefix, prob.total_suffix, prob.h_q, prob.h_kv,
            prob.head_dim)
    bufs["ws_f"] = torch.empty(binding.workspace_bytes("fwd", *args), device="cuda", dtype=torch.uint8)
    bufs["ws_b"] = torch.empty(binding.workspace_bytes("bwd", *args), device="cuda", dtype=torch.uint8)
    return bufs


def time_last(binding, torch, dev, prob, steps, warmup):
    """The final-token forward (every member's last query only) on this workload.

    HBM-bound: the algorithmic traffic is every key and value row read once, the members' final query rows
    read once, and their outputs (and fp32 log-sum-exp) written once; the matrix work is a few GFLOP.
    """
    ns = len(prob.suffix_lens)
    el = 2 if prob.dtype == "bf16" else 4
    names = ("q_pre", "k_pre", "v_pre", "q_suf", "k_suf", "v_suf")
    outs = (torch.empty((ns, prob.h_q, prob.head_dim), device="cuda", dtype=dev["q_pre"].dtype),
            torch.empty((prob.h_q, ns), device="cuda", dtype=torch.float32))
    nbytes_ws = int(binding.lib().pg_attn_fwd_last_workspace_size(len(prob.prefix_lens), ns, prob.total_prefix,
                                                                  prob.total_suffix, prob.h_q, prob.h_kv,
                                                                  prob.head_dim))
    ws = torch.empty(nbytes_ws, device="cuda", dtype=torch.uint8)
    call = lambda: binding.fwd_last(*[dev[n] for n in names], dev["cu_prefix"], dev["cu_suffix"],  # noqa: E731
                                    dev["group_sizes"], dev["scale"], out=outs, workspace=ws)
    for _ in range(warmup):
        call()
    torch.cuda.synchronize()
    binding.timing_start()
    for _ in range(steps):
        call()
    torch.cuda.synchronize()
    binding.timing_stop()
    n, tot = binding.timing_get("last")
    ms = tot / n
    rows = prob.total_prefix + prob.total_suffix
    nbytes = 2 * rows * prob.h_kv * prob.head_dim * el + 2 * ns * prob.h_q * prob.head_dim * el + ns * prob.h_q * 4
    gbs = nbytes / (ms * 1e-3) / 1e9
    return {"kernel": "last (+ merge)", "ms": round(ms, 4), "bytes": nbytes, "achieved_GBps": round(gbs, 1),
            "peak_GBps": 8000.0, "frac": round(gbs / 8000.0, 4), "bound": "hbm", "queries": ns * prob.h_q}


def time_rope(binding, torch, dev, prob, steps, warmup):
    """The grouped-position rotary embedding of q and k (both sides) on this workload, out of place.

    HBM-bound: every element of q and k is read once and written once, so the algorithmic traffic of one
    launch is 2 * (total_prefix + total_suffix) * (h_q + h_kv) * head_dim * element bytes; the HBM peak is
    8 TB/s.
    """
    ins = (dev["q_pre"], dev["q_suf"], dev["k_pre"], dev["k_suf"])
    outs = tuple(torch.empty_like(t) for t in ins)
    ws = torch.empty(int(binding.lib().pg_rope_workspace_size(len(prob.prefix_lens))), device="cuda",
                     dtype=torch.uint8)
    grp = (dev["cu_prefix"], dev["cu_suffix"], dev["group_sizes"])
    for _ in range(warmup):
        binding.rope(*ins, *grp, out=outs, workspace=ws)
    torch.cuda.synchronize()
    binding.timing_start()
    for _ in range(steps):
        binding.rope(*ins, *grp, out=outs, workspace=ws)
    torch.cuda.synchronize()
    binding.timing_stop()
    n, tot = binding.timing_get("rope")
    ms = tot / n
    el = 2 if prob.dtype == "bf16" else 4
    nbytes = 2 * (prob.total_prefix + prob.total_suffix) * (prob.h_q + prob.h_kv) * prob.head_dim * el
    gbs = nbytes / (ms * 1e-3) / 1e9
    return {"kernel": "rope", "ms": round(ms, 4), "bytes": nbytes, "achieved_GBps": round(gbs, 1),
            "peak_GBps": 8000.0, "frac": round(gbs / 8000.0, 4), "bound": "hbm"}


def cpu_baseline(prob, useful_per_pair_head, budget_s):
    """The oracle (fp64 numpy, as it stands) on a bounded sample of the workload.

    The sample is all rows and members of the first k query heads, fwd+bwd; one head is
    timed first and k is chosen so the measured run takes about ``budget_s`` seconds.
    """
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import grouped_oracle
    t = {k: prob.as_float(k, np.float64) for k in prob.tensors}
    pairs_rep = repeated_pair_count(prob.prefix_lens, prob.group_sizes, prob.suffix_lens)
    pairs = pair_count(prob.prefix_lens, prob.group_sizes, prob.suffix_lens)

    def run(n):
        t0 = time.perf_counter()
        grouped_oracle(prob.prefix_lens, prob.group_sizes, prob.suffix_lens, t, prob.scale, grads=True,
                       heads=list(range(n)), check_members=False)
        return time.perf_counter() - t0

    dt1 = run(1)
    n_heads = max(1, min(prob.h_q, round(budget_s / max(dt1, 1e-3))))
    dt = run(n_heads) if n_heads > 1 else dt1
    useful = useful_per_pair_head * pairs * n_heads
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    return {"value": useful / dt / 1e12, "unit": "TFLOP/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{n_heads} of {prob.h_q} query heads, all rows and members, fp64 numpy, repeated-prefix "
                      f"({pairs_rep} repeated pairs per head), fwd+bwd; {dt:.1f} s",
            "seconds": round(dt, 2), "host_cpus": len(os.sched_getaffinity(0))}


ATTN_SOURCES = ("pg_attn.hip", "pg_bwd.hpp", "pg_common.hpp", "pg_fwd.hpp", "pg_plan.hpp")


def kernel_source_sha():
    """Digest of the sources the attention kernels and their launches are built from: counter readings are
    only reported for the build they were taken on."""
    h = hashlib.sha256()
    for name in ATTN_SOURCES:
        f = os.path.join(ROOT, "paper_2506_05433_amd", "csrc", name)
        with open(f, "rb") as fh:
            h.update(os.path.basename(f).encode() + b"\0" + fh.read())
    return h.hexdigest()[:16]


def recorded_traffic(kernel, workload):
    """HBM bytes per launch from profiles/traffic_<kernel>_<workload>.json if taken on this source, else None.

    The file holds rocprofv3 FETCH_SIZE and WRITE_SIZE (KiB per dispatch) of the kernel and of a plain
    device copy of known size; each counter is scaled by copy_bytes / counter(copy).
    """
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        t = json.load(fh)
    if t.get("source_sha") != kernel_source_sha():
        return None
    f = t["fetch_kib"] * t["copy_read_bytes"] / t["copy_fetch_kib"]
    w = t["write_kib"] * t["copy_write_bytes"] / t["copy_write_kib"]
    return f + w


def calibrate_copy(n_bytes):
    """A plain device-to-device copy of n_bytes (reference reading for the HBM byte counters)."""
    import torch
    src = torch.empty(n_bytes // 4, device="cuda", dtype=torch.float32).fill_(1.0)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": n_bytes, "launches": 3}))


def tensor_bytes(prob, grads=True):
    """Device bytes of the layer's tensors for one layout (inputs, outputs, LSE and, with grads, dO and dQ/dK/dV)."""
    el = 2 if prob.dtype == "bf16" else 4
    rows = prob.total_prefix + prob.total_suffix
    per_row = (2 * prob.h_q + 2 * prob.h_kv) * prob.head_dim * el + prob.h_q * 4  # q, o, k, v, lse
    if grads:
        per_row += (2 * prob.h_q + 2 * prob.h_kv) * prob.head_dim * el  # do, dq, dk, dv
    return rows * per_row


def sweep(args):
    """Fig. 2/3 grid of the paper: prefix 4096/8192/16384, G in {2,4,8,16}, prefix/response ratio r.

    Every member has the same response length P / r (the setting of Appendix A.2). For each point the
    grouped and the repeated layouts run the same kernels; the line reports both times, the speedup,
    Eq. (17)'s attention-cost ratio, the useful TFLOP/s and the tensor + workspace bytes of both layouts.
    """
    import torch

    from paper_2506_05433_amd import binding
    from paper_2506_05433_amd.inputs import Workload, make_problem, repeated_layout
    rows = []
    for P in (4096, 8192, 16384):
        for G in (2, 4, 8, 16):
            for r in (1, 4, 16):
                S = P // r
                wl = Workload(f"sweep_P{P}_G{G}_r{r}", 1, G, ("fixed", P), ("uniform", S, S), 32, 8, 128, "bf16",
                              1.0 / 128 ** 0.5)
                prob = make_problem(wl, seed=0)
                pairs = pair_count(prob.prefix_lens, prob.group_sizes, prob.suffix_lens)
                flops = 14.0 * 128 * 32 * pairs
                out = {"P": P, "G": G, "r": r, "S": S}
                for name, pr in (("grouped", prob), ("repeated", repeated_layout(prob))):
                    # names the case before any GPU work on it, on stdout
                    print(f"[sweep] P={P} G={G} r={r} {name}: groups={len(pr.prefix_lens)} "
                          f"total_prefix={pr.total_prefix} total_suffix={pr.total_suffix}", flush=True)
                    dev = binding.to_device(pr, "cuda")
                    bufs = alloc(binding, torch, dev, pr)
                    ms, _, _ = time_steps(binding, torch, dev, bufs, args.steps, args.warmup)
                    ws = sum(b.numel() for b in (bufs["ws_f"], bufs["ws_b"]))
                    out[name + "_ms"] = round(ms, 4)
                    out[name + "_MB"] = round((tensor_bytes(pr) + ws) / 1e6, 1)
                    del dev, bufs
                    torch.cuda.empty_cache()
                eq17 = (P * P + G * S * (2 * P + S)) / (G * (P + S) ** 2)
                out.update({"speedup": round(out["repeated_ms"] / out["grouped_ms"], 3),
                            "eq17_cost_ratio": round(eq17, 4), "eq17_speedup": round(1 / eq17, 3),
                            "useful_tflops": round(flops / (out["grouped_ms"] * 1e-3) / 1e12, 1),
                            "memory_ratio": round(out["grouped_MB"] / out["repeated_MB"], 3)})
                print(json.dumps(out), flush=True)
                rows.append(out)
    return rows


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="single_group")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-repeated", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=20.0)
    ap.add_argument("--sweep", action="store_true",
                    help="run the paper's Fig. 2/3 grid (one JSON line per point) instead of the bench line")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="BYTES",
                    help="only run a plain device copy of BYTES (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: this build has no multi-GPU path (asked for --gpus {args.gpus}).",
              file=sys.stderr)
        sys.exit(2)

    if args.calibrate_copy:
        calibrate_copy(args.calibrate_copy)
        return
    if args.sweep:
        sweep(args)
        return

    import torch

    from paper_2506_05433_amd import binding
    from paper_2506_05433_amd.inputs import WORKLOADS, make_problem, repeated_layout

    wl = WORKLOADS[args.workload]
    progress(f"{wl.name}: generating inputs")
    prob = make_problem(wl, seed=0)
    d, hq = prob.head_dim, prob.h_q
    pairs = pair_count(prob.prefix_lens, prob.group_sizes, prob.suffix_lens)
    rep_pairs = repeated_pair_count(prob.prefix_lens, prob.group_sizes, prob.suffix_lens)
    fwd_flops = 4.0 * d * hq * pairs
    bwd_flops = 10.0 * d * hq * pairs
    dev = binding.to_device(prob, "cuda")
    bufs = alloc(binding, torch, dev, prob)
    print(f"[bench] {wl.name}: pairs={pairs} tokens={prob.total_prefix + prob.total_suffix}", file=sys.stderr,
          flush=True)
    ms, kern, ms_eager = time_steps(binding, torch, dev, bufs, args.steps, args.warmup)
    progress(f"grouped layout: {ms:.3f} ms/step")
    value = (fwd_flops + bwd_flops) / (ms * 1e-3) / 1e12
    peak = PEAK_TFLOPS[prob.dtype]
    algo = {"fwd": fwd_flops, "dkdv": 8.0 * d * hq * pairs, "dq": 6.0 * d * hq * pairs}
    dom = max(("fwd", "dkdv", "dq"), key=lambda k: (kern[k]["avg_ms"] or 0.0))
    achieved = algo[dom] / (kern[dom]["avg_ms"] * 1e-3) / 1e12
    fwd_ms = kern["fwd"]["avg_ms"]
    bwd_ms = sum(kern[k]["avg_ms"] or 0.0 for k in ("dkdv", "dq"))
    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": prob.dtype, "data": "synthetic (seeded normal inputs, lengths drawn per workload)",
        "config": {"workload": wl.name, "desc": wl.note, "n_groups": int(len(prob.prefix_lens)),
                   "total_prefix": prob.total_prefix, "total_suffix": prob.total_suffix, "h_q": hq,
                   "h_kv": prob.h_kv, "head_dim": d, "pairs": pairs, "parallelism": "single GPU"},
        "ms_per_step_eager": round(ms_eager, 4), "step": "one HIP-graph replay of fwd+bwd (eager launches: "
                                                         "ms_per_step_eager)",
        "pct_of_peak": round(100.0 * value / peak, 2),
        "fwd_tflops": round(fwd_flops / (fwd_ms * 1e-3) / 1e12, 2) if fwd_ms else None,
        "bwd_tflops": round(bwd_flops / (bwd_ms * 1e-3) / 1e12, 2) if bwd_ms else None,
        "kernels_ms": {k: (round(v["avg_ms"], 4) if v["avg_ms"] else None) for k, v in kern.items()},
        "roofline": {"bound": "mfma", "kernel": dom, "achieved": round(achieved, 2), "peak": peak,
                     "unit": "TFLOP/s", "frac": round(achieved / peak, 4),
                     "traffic": recorded_traffic(dom, wl.name), "source_sha": kernel_source_sha()},
    }
    out["rope"] = time_rope(binding, torch, dev, prob, args.steps, args.warmup)
    out["last"] = time_last(binding, torch, dev, prob, args.steps, args.warmup)
    if not args.no_repeated:
        progress("building the repeated-prefix layout")
        rep = repeated_layout(prob)
        del dev, bufs
        torch.cuda.empty_cache()
        rdev = binding.to_device(rep, "cuda")
        rbufs = alloc(binding, torch, rdev, rep)
        rms, _, _ = time_steps(binding, torch, rdev, rbufs, args.steps, args.warmup)
        progress(f"repeated layout: {rms:.3f} ms/step")
        G = prob.group_sizes
        P = prob.prefix_lens
        sum_s = prob.suffix_lens.sum()
        target = 0.8 * float((G * P).sum() + sum_s) / float(P.sum() + sum_s)
        out.update({"repeated_ms_per_step": round(rms, 4), "speedup_vs_repeated": round(rms / ms, 3),
                    "speedup_target": round(target, 3), "speedup_ceiling_pairs": round(rep_pairs / pairs, 3)})
        del rdev, rbufs
    if not args.no_cpu_baseline:
        progress("timing the CPU oracle on a sample")
        out["cpu_baseline"] = cpu_baseline(prob, 14.0 * d, args.cpu_budget)
    print(json.dumps(out))


if __name__ == "__main__":
    main()

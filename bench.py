"""Benchmark: grouped (shared-prefix) attention forward+backward on one MI355X.

python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--padded]
                [--no-cpu-baseline] [--no-repeated] [--sweep]

A step is one forward and one backward call over the whole workload (inputs
resident in HBM). The default workload is the largest one, ``packed_varlen``
(8 groups, G=16, prefix lengths log-uniform in [1024, 32768], responses
uniform in [64, 4096], 64/8 heads, d=128, bf16). Prints ONE JSON line.

``value`` is useful TFLOP/s: 4*d*H_q*pairs (forward) + 10*d*H_q*pairs
(backward) per step, where pairs is the exact number of (query, key) pairs the
grouped problem allows; masked work, ragged tiles and the repeated-prefix
pairs the method avoids are not counted.

Timing protocol: W untimed warmup steps, then K timed steps. Before every
timed step a 512 MiB buffer is overwritten (evicting the 256 MB Infinity
Cache), and each step is bracketed by its own HIP events on the stream the
library launches on; ``ms_per_step`` is the median. The timed step is the
forward and backward calls captured once as a HIP graph and replayed; the
same protocol on eager launches gives ``ms_per_step_eager`` and, through the
library's own per-launch events, the per-kernel averages. The same kernels are
timed on the repeated-prefix layout (every member with its own copy of the
prefix; and with ``--padded`` also every member padded to the group's longest
response, Eq. (1)) for the speedup.
"""
import argparse
import hashlib
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "grouped attn fwd+bwd TFLOP/s (useful) & % MFMA peak; speedup vs repeated-prefix"
PEAK_TFLOPS = {"bf16": 2500.0, "fp32": 157.3}
DEFAULT_WORKLOAD = "packed_varlen"
FLUSH_BYTES = 512 << 20


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


def padded_pair_count(prefix_lens, group_sizes, suffix_lens):
    """Pairs of the padded layout of Eq. (1): every member of a group padded to its longest response."""
    total, m = 0, 0
    for p, g in zip(prefix_lens, group_sizes):
        g = int(g)
        if g:
            n = int(p) + int(max(suffix_lens[m:m + g]))
            total += g * (n * (n + 1) // 2)
        m += g
    return total


def progress(msg):
    """A progress line on stderr (the JSON result is the only stdout line)."""
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


class Flusher:
    """Overwrites a 512 MiB device buffer: run before each timed step so that no operand is served from the
    256 MB Infinity Cache (or the L2s) left warm by the previous step."""

    def __init__(self, torch):
        self.buf = torch.empty(FLUSH_BYTES // 4, device="cuda", dtype=torch.float32)
        self.k = 0

    def __call__(self):
        self.k += 1
        self.buf.fill_(float(self.k & 7))


def step_fn(binding, dev, bufs):
    def step():
        binding.fwd(dev["q_pre"], dev["k_pre"], dev["v_pre"], dev["q_suf"], dev["k_suf"], dev["v_suf"],
                    dev["cu_prefix"], dev["cu_suffix"], dev["group_sizes"], dev["scale"], out=bufs["fwd"],
                    workspace=bufs["ws_f"])
        o_pre, o_suf, lse_pre, lse_suf = bufs["fwd"]
        binding.bwd(dev["q_pre"], dev["k_pre"], dev["v_pre"], dev["q_suf"], dev["k_suf"], dev["v_suf"],
                    o_pre, o_suf, lse_pre, lse_suf, dev["do_pre"], dev["do_suf"],
                    dev["cu_prefix"], dev["cu_suffix"], dev["group_sizes"], dev["scale"], out=bufs["bwd"],
                    workspace=bufs["ws_b"])
    return step


def timed_steps(torch, run, steps, flush, label):
    """Per-step GPU times (ms) of ``run`` over ``steps`` steps, each after a cache flush and bracketed by its
    own events on the current stream; the host waits for each step (progress lines every ~20 s)."""
    times = []
    t_last = time.monotonic()
    for i in range(steps):
        flush()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        run()
        e1.record()
        e1.synchronize()
        times.append(e0.elapsed_time(e1))
        if time.monotonic() - t_last > 20.0:
            progress(f"{label}: step {i + 1}/{steps}, median so far {statistics.median(times):.3f} ms")
            t_last = time.monotonic()
    return times


def time_layout(binding, torch, dev, bufs, steps, warmup, flush, label, eager=True):
    """Graph-replay (and optionally eager) step times of one layout; per-kernel averages from the eager pass."""
    step = step_fn(binding, dev, bufs)
    out = {}
    if eager:
        for _ in range(warmup):
            step()
        torch.cuda.synchronize()
        binding.timing_start()
        times = timed_steps(torch, step, steps, flush, label + " (eager)")
        torch.cuda.synchronize()
        binding.timing_stop()
        out["eager_ms"] = times
        kern = {}
        for k in ("plan", "fwd", "dq", "dkdv", "kv_reduce"):
            n, tot = binding.timing_get(k)
            kern[k] = (tot / n) if n else None
        out["kernels_ms"] = kern
    else:
        step()
        torch.cuda.synchronize()
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
    out["graph_ms"] = timed_steps(torch, graph.replay, steps, flush, label)
    del graph
    return out


def alloc(binding, torch, dev, prob_shape):
    """Outputs and workspaces of one layout. ``prob_shape`` = (n_groups, n_suffixes, total_prefix,
    total_suffix, h_q, h_kv, head_dim)."""
    ng, ns, tp, ts, hq, hkv, d = prob_shape
    bufs = {
        "fwd": (torch.empty_like(dev["q_pre"]), torch.empty_like(dev["q_suf"]),
                torch.empty((hq, tp), device="cuda", dtype=torch.float32),
                torch.empty((hq, ts), device="cuda", dtype=torch.float32)),
        "bwd": tuple(torch.empty_like(dev[k]) for k in ("q_pre", "k_pre", "v_pre", "q_suf", "k_suf", "v_suf")),
    }
    bufs["ws_f"] = torch.empty(binding.workspace_bytes("fwd", *prob_shape), device="cuda", dtype=torch.uint8)
    bufs["ws_b"] = torch.empty(binding.workspace_bytes("bwd", *prob_shape), device="cuda", dtype=torch.uint8)
    return bufs


def copy_sum_fn(torch, prob, bufs):
    """The step a repeated-layout trainer adds after its backward to recover the shared prefix's gradients: the
    G-way sum of each group's prefix copies of dQ, dK and dV (timed apart from the kernels, on the device)."""
    segs, row = [], 0
    for p, gs in zip(prob.prefix_lens, prob.group_sizes):
        p, gs = int(p), int(gs)
        if gs > 1 and p > 0:
            segs.append((row, gs, p))
        row += max(gs, 1) * p
    grads = bufs["bwd"][:3]  # dq_pre, dk_pre, dv_pre of the repeated layout
    outs = [[torch.empty((p,) + tuple(t.shape[1:]), device=t.device, dtype=t.dtype) for (_, _, p) in segs]
            for t in grads]

    def run():
        for t, o in zip(grads, outs):
            for (r0, gs, p), dst in zip(segs, o):
                torch.sum(t[r0:r0 + gs * p].view(gs, p, *t.shape[1:]), dim=0, out=dst)
    run.outs = outs  # [gradient][group with copies]
    return run


def shape_of(prob):
    return (len(prob.prefix_lens), len(prob.suffix_lens), prob.total_prefix, prob.total_suffix, prob.h_q,
            prob.h_kv, prob.head_dim)


def baseline_layout(torch, dev, prob, padded, copy=False):
    """The repeated-prefix layout (Eq. (1) without padding), or with ``padded`` the padded one (every member's
    response padded with zero rows to the group's longest), built on the device from the grouped tensors.

    Every member becomes a group of size 1 holding its own copy of the group's prefix; ``do_pre`` goes whole
    to a group's first copy and zero to the others, so the copies' summed prefix gradients equal the grouped
    ones. Groups with no members keep their prefix as a group of size 0. The unpadded layout shares the
    response tensors with ``dev`` unless ``copy`` (so that a memory measurement counts them). Returns (device
    dict, shape)."""
    import numpy as np
    cu_p, cu_s = prob.cu_prefix, prob.cu_suffix
    pre_idx, zero_do, prefix, groups, suffix, suf_src = [], [], [], [], [], []
    m, row = 0, 0
    for g, (p, gs) in enumerate(zip(prob.prefix_lens, prob.group_sizes)):
        p, gs = int(p), int(gs)
        rows = np.arange(cu_p[g], cu_p[g + 1])
        width = int(max(prob.suffix_lens[m:m + gs])) if (gs and padded) else 0
        for i in range(max(gs, 1)):
            pre_idx.append(rows)
            if i > 0:
                zero_do.append(np.arange(row, row + p))
            row += p
            prefix.append(p)
            groups.append(1 if gs else 0)
            if gs:
                s = int(prob.suffix_lens[m + i])
                n = width if padded else s
                src = np.full(n, -1, np.int64)
                src[:s] = np.arange(cu_s[m + i], cu_s[m + i + 1])
                suf_src.append(src)
                suffix.append(n)
        m += gs
    cat = lambda xs: np.concatenate(xs) if xs else np.zeros(0, np.int64)  # noqa: E731
    pre_idx, zero_do, suf_src = cat(pre_idx), cat(zero_do), cat(suf_src)
    out = {}
    where = dev["q_pre"].device
    ipre = torch.from_numpy(pre_idx).to(where)
    for name in ("q_pre", "k_pre", "v_pre", "do_pre"):
        out[name] = dev[name].index_select(0, ipre)
    if zero_do.size:
        out["do_pre"].index_fill_(0, torch.from_numpy(zero_do).to(where), 0)
    if padded:
        # padding rows read row 0 and are then zeroed
        isuf = torch.from_numpy(np.maximum(suf_src, 0)).to(where)
        pad = torch.from_numpy(np.nonzero(suf_src < 0)[0]).to(where)
        for name in ("q_suf", "k_suf", "v_suf", "do_suf"):
            t = dev[name].index_select(0, isuf)
            if pad.numel():
                t.index_fill_(0, pad, 0)
            out[name] = t
    else:
        for name in ("q_suf", "k_suf", "v_suf", "do_suf"):
            out[name] = dev[name].clone() if copy else dev[name]
    i32 = lambda a: torch.from_numpy(np.asarray(a, np.int32)).to(where)  # noqa: E731
    out["cu_prefix"] = i32(np.concatenate([[0], np.cumsum(prefix)]))
    out["cu_suffix"] = i32(np.concatenate([[0], np.cumsum(suffix)]))
    out["group_sizes"] = i32(groups)
    out["scale"] = prob.scale
    shape = (len(prefix), len(suffix), int(sum(prefix)), int(sum(suffix)), prob.h_q, prob.h_kv, prob.head_dim)
    return out, shape


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


def time_xours(binding, torch, dev, prob, steps, warmup, flush, split_ms):
    """The same fwd+bwd step through the single-buffer calls of Eq. (2) (pg_attn_fwd_xours / pg_attn_bwd_xours):
    every tensor one buffer holding, group after group, the prefix rows and then the members' response rows.
    Timed like the headline (median of cache-flushed HIP-graph replays); same kernels, so the ratio to the
    split-buffer step should be ~1."""
    from paper_2506_05433_amd.inputs import xours_order
    tp = prob.total_prefix
    idx = torch.from_numpy(xours_order(prob)).to(dev["q_pre"].device)
    x = {n: torch.cat([dev[n + "_pre"], dev[n + "_suf"]]).index_select(0, idx) for n in ("q", "k", "v", "do")}
    grp = (dev["cu_prefix"], dev["cu_suffix"], dev["group_sizes"], tp, dev["scale"])
    rows = x["q"].shape[0]
    fo = (torch.empty_like(x["q"]), torch.empty((prob.h_q, rows), device="cuda", dtype=torch.float32))
    bo = (torch.empty_like(x["q"]), torch.empty_like(x["k"]), torch.empty_like(x["v"]))
    shape = shape_of(prob)
    ws_f = torch.empty(binding.workspace_bytes("fwd", *shape), device="cuda", dtype=torch.uint8)
    ws_b = torch.empty(binding.workspace_bytes("bwd", *shape), device="cuda", dtype=torch.uint8)

    def step():
        binding.fwd_xours(x["q"], x["k"], x["v"], *grp, out=fo, workspace=ws_f)
        binding.bwd_xours(x["q"], x["k"], x["v"], fo[0], fo[1], x["do"], *grp, out=bo, workspace=ws_b)
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
    ms = statistics.median(timed_steps(torch, graph.replay, steps, flush, "single-buffer layout"))
    del graph, x, fo, bo, ws_f, ws_b
    torch.cuda.empty_cache()
    return {"ms_per_step": round(ms, 4), "vs_split_layout": round(split_ms / ms, 3)}


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
    del outs
    return {"kernel": "rope", "ms": round(ms, 4), "bytes": nbytes, "achieved_GBps": round(gbs, 1),
            "peak_GBps": 8000.0, "frac": round(gbs / 8000.0, 4), "bound": "hbm"}


def sub_problem(prob, g, h):
    """Group g and query head h of ``prob`` as a problem of its own (one query head and its key/value head),
    decoded to float64: the unit the CPU oracle is timed on."""
    import numpy as np
    cu_p, cu_s = prob.cu_prefix, prob.cu_suffix
    m0 = int(prob.group_sizes[:g].sum())
    m1 = m0 + int(prob.group_sizes[g])
    p0, p1, s0, s1 = int(cu_p[g]), int(cu_p[g + 1]), int(cu_s[m0]), int(cu_s[m1])
    kv = h // (prob.h_q // prob.h_kv)
    t = {}
    for name, a in prob.tensors.items():
        rows = slice(p0, p1) if name.endswith("_pre") else slice(s0, s1)
        hs = slice(kv, kv + 1) if name[0] in "kv" else slice(h, h + 1)
        a = np.ascontiguousarray(a[rows, hs])
        if a.dtype == np.uint16:
            a = (a.astype(np.uint32) << 16).view(np.float32)
        t[name] = a.astype(np.float64)
    lengths = (np.array([p1 - p0]), np.array([m1 - m0]), np.asarray(prob.suffix_lens[m0:m1]))
    return lengths, t


def cpu_baseline(prob, budget_s):
    """The oracle (fp64 numpy, as it stands) on a bounded sample of the workload: whole (group, query head)
    units, fwd+bwd, timed one call at a time.

    The smallest group's first head is timed first; that rate picks the group by work rank (the median
    group, or a smaller one if one of its heads would take more than ~40 s), whose heads then run until the
    budget is spent. ``value`` = useful flops of the units run (14*d per grouped pair and head, as for the
    GPU) / their total time."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import grouped_oracle
    ng = len(prob.prefix_lens)
    cs = np.concatenate([[0], np.cumsum(prob.group_sizes)])
    per_group = []
    for g in range(ng):
        lens = ([prob.prefix_lens[g]], [prob.group_sizes[g]], prob.suffix_lens[cs[g]:cs[g + 1]])
        per_group.append((repeated_pair_count(*lens), pair_count(*lens)))
    order = [g for g in sorted(range(ng), key=lambda g: per_group[g][0]) if per_group[g][0] > 0]
    useful_per_pair = 14.0 * prob.head_dim
    units, total_s, total_flops = [], 0.0, 0.0

    def run(g, h):
        nonlocal total_s, total_flops
        lengths, t = sub_problem(prob, g, h)
        t0 = time.perf_counter()
        grouped_oracle(*lengths, t, prob.scale, grads=True, check_members=False)
        dt = time.perf_counter() - t0
        total_s += dt
        total_flops += useful_per_pair * per_group[g][1]
        units.append((g, h))
        progress(f"cpu oracle: group {g} head {h}: {dt:.1f} s")
        return dt

    if not order:
        return None
    g0 = order[0]
    rate = per_group[g0][0] / max(run(g0, 0), 1e-6)  # repeated pairs per second
    cand = [g for g in order if per_group[g][0] / rate <= min(40.0, budget_s)]
    g1 = cand[min(len(cand) - 1, len(order) // 2)] if cand else g0
    h = 0 if g1 != g0 else 1
    while h < prob.h_q and total_s + per_group[g1][0] / rate <= budget_s:
        run(g1, h)
        h += 1
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    desc = ", ".join(f"g{g}h{h}" for g, h in units)
    return {"value": total_flops / total_s / 1e12, "unit": "TFLOP/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{len(units)} (group, query head) units [{desc}] of {ng} groups x {prob.h_q} heads "
                      f"(groups P={[int(prob.prefix_lens[g]) for g in sorted(set(u[0] for u in units))]}), "
                      f"all rows and members of each, fp64 numpy, repeated-prefix, fwd+bwd; {total_s:.1f} s",
            "seconds": round(total_s, 2), "host_cpus": len(os.sched_getaffinity(0)), "cpu_model": cpu_model()}


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


ATTN_SOURCES = ("pg_attn.hip", "pg_bwd.hpp", "pg_common.hpp", "pg_fwd.hpp", "pg_plan.hpp", "pg_types.hpp")


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


def recorded_trace_us(kernel, workload):
    """Average duration (us) of ``kernel`` from the rocprofv3 kernel-trace summary
    profiles/trace_<workload>.json, if taken on this source, else None."""
    path = os.path.join(ROOT, "profiles", f"trace_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        t = json.load(fh)
    if t.get("source_sha") != kernel_source_sha():
        return None
    return t.get("avg_us", {}).get(kernel)


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


def measured_peak_bytes(torch, build):
    """Peak device bytes allocated while ``build()`` allocates a layout and runs one fwd+bwd step on it,
    above what was allocated before (torch's allocator statistics; the library allocates nothing)."""
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    base = torch.cuda.memory_allocated()
    torch.cuda.reset_peak_memory_stats()
    keep = build()
    torch.cuda.synchronize()
    peak = torch.cuda.max_memory_allocated() - base
    return peak, keep


def sweep(args):
    """Fig. 2/3 grid of the paper: prefix 4096/8192/16384, G in {2,4,8,16}, prefix/response ratio r.

    Member i's response length is drawn uniform in [S/2, 3S/2] with S = P / r (the ratio is prefix over mean
    response), so the padded layout of Eq. (1) differs from the unpadded repeated one. For each point the
    grouped, repeated and padded layouts run the same kernels; the line reports the three times, the
    speedups, Eq. (17)'s attention-cost ratio at the mean lengths, the useful TFLOP/s, and each layout's
    measured peak device memory for one fwd+bwd step (inputs, outputs, gradients and workspaces).
    """
    import torch

    from paper_2506_05433_amd import binding
    from paper_2506_05433_amd.inputs import Workload, make_problem
    flush = Flusher(torch)
    rows = []
    for P in (4096, 8192, 16384):
        for G in (2, 4, 8, 16):
            for r in (1, 4, 16):
                S = P // r
                wl = Workload(f"sweep_P{P}_G{G}_r{r}", 1, G, ("fixed", P), ("uniform", S // 2, S + S // 2), 32, 8,
                              128, "bf16", 1.0 / 128 ** 0.5)
                prob = make_problem(wl, seed=0)
                pairs = pair_count(prob.prefix_lens, prob.group_sizes, prob.suffix_lens)
                flops = 14.0 * 128 * 32 * pairs
                out = {"P": P, "G": G, "r": r, "S_mean": S, "S": [int(x) for x in prob.suffix_lens]}
                for name in ("grouped", "repeated", "padded"):
                    # names the case before any GPU work on it
                    print(f"[sweep] P={P} G={G} r={r} {name}", flush=True)
                    # the baselines are gathered from the grouped tensors, which are allocated before the
                    # measured region; each layout's peak counts its own inputs, outputs, gradients and
                    # workspaces
                    src = binding.to_device(prob, "cuda") if name != "grouped" else None

                    def build():
                        if name == "grouped":
                            dev, shape = binding.to_device(prob, "cuda"), shape_of(prob)
                        else:
                            dev, shape = baseline_layout(torch, src, prob, padded=name == "padded", copy=True)
                        bufs = alloc(binding, torch, dev, shape)
                        step_fn(binding, dev, bufs)()
                        return dev, bufs

                    peak, (dev, bufs) = measured_peak_bytes(torch, build)
                    del src
                    res = time_layout(binding, torch, dev, bufs, args.steps, args.warmup, flush, name, eager=False)
                    out[name + "_ms"] = round(statistics.median(res["graph_ms"]), 4)
                    out[name + "_peak_MB"] = round(peak / 1e6, 1)
                    del dev, bufs
                    torch.cuda.empty_cache()
                Lr = S
                eq17 = (P * P + G * Lr * (2 * P + Lr)) / (G * (P + Lr) ** 2)
                out.update({"speedup_vs_repeated": round(out["repeated_ms"] / out["grouped_ms"], 3),
                            "speedup_vs_padded": round(out["padded_ms"] / out["grouped_ms"], 3),
                            "eq17_cost_ratio": round(eq17, 4), "eq17_speedup": round(1 / eq17, 3),
                            "pair_ratio_repeated": round(repeated_pair_count(prob.prefix_lens, prob.group_sizes,
                                                                             prob.suffix_lens) / pairs, 3),
                            "pair_ratio_padded": round(padded_pair_count(prob.prefix_lens, prob.group_sizes,
                                                                         prob.suffix_lens) / pairs, 3),
                            "useful_tflops": round(flops / (out["grouped_ms"] * 1e-3) / 1e12, 1),
                            "memory_ratio_repeated": round(out["grouped_peak_MB"] / out["repeated_peak_MB"], 3),
                            "memory_ratio_padded": round(out["grouped_peak_MB"] / out["padded_peak_MB"], 3)})
                print(json.dumps(out), flush=True)
                rows.append(out)
    return rows


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-repeated", action="store_true")
    ap.add_argument("--padded", action="store_true", help="also time the padded layout of Eq. (1)")
    ap.add_argument("--no-extras", action="store_true", help="skip the rotary-embedding and final-token timings")
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
    from paper_2506_05433_amd.inputs import WORKLOADS, make_problem

    wl = WORKLOADS[args.workload]
    progress(f"{wl.name}: generating inputs")
    t0 = time.monotonic()
    prob = make_problem(wl, seed=0)
    d, hq = prob.head_dim, prob.h_q
    pairs = pair_count(prob.prefix_lens, prob.group_sizes, prob.suffix_lens)
    rep_pairs = repeated_pair_count(prob.prefix_lens, prob.group_sizes, prob.suffix_lens)
    fwd_flops = 4.0 * d * hq * pairs
    bwd_flops = 10.0 * d * hq * pairs
    progress(f"{wl.name}: pairs={pairs} tokens={prob.total_prefix + prob.total_suffix} "
             f"(inputs drawn in {time.monotonic() - t0:.0f} s)")
    flush = Flusher(torch)
    dev = binding.to_device(prob, "cuda")
    bufs = alloc(binding, torch, dev, shape_of(prob))
    res = time_layout(binding, torch, dev, bufs, args.steps, args.warmup, flush, "grouped")
    ms = statistics.median(res["graph_ms"])
    ms_eager = statistics.median(res["eager_ms"])
    kern = res["kernels_ms"]
    progress(f"grouped layout: {ms:.3f} ms/step (median of {args.steps})")
    value = (fwd_flops + bwd_flops) / (ms * 1e-3) / 1e12
    peak = PEAK_TFLOPS[prob.dtype]
    algo = {"fwd": fwd_flops, "dkdv": 8.0 * d * hq * pairs, "dq": 6.0 * d * hq * pairs}
    dom = max(("fwd", "dkdv", "dq"), key=lambda k: (kern[k] or 0.0))
    achieved = algo[dom] / (kern[dom] * 1e-3) / 1e12
    fwd_ms = kern["fwd"]
    bwd_ms = sum(kern[k] or 0.0 for k in ("dkdv", "dq", "kv_reduce"))
    roof = {"bound": "mfma", "kernel": dom, "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
            "frac": round(achieved / peak, 4), "traffic": recorded_traffic(dom, wl.name),
            "algorithmic_flops": algo[dom], "avg_ms_events": round(kern[dom], 4),
            "source_sha": kernel_source_sha()}
    tr = recorded_trace_us(dom, wl.name)
    if tr:
        roof["avg_ms_trace"] = round(tr / 1e3, 4)
        roof["frac_trace"] = round(algo[dom] / (tr * 1e-6) / 1e12 / peak, 4)
    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": prob.dtype,
        "data": "synthetic (seeded normal inputs, lengths drawn per workload)",
        "config": {"workload": wl.name, "desc": wl.note, "n_groups": int(len(prob.prefix_lens)),
                   "total_prefix": prob.total_prefix, "total_suffix": prob.total_suffix, "h_q": hq,
                   "h_kv": prob.h_kv, "head_dim": d, "pairs": pairs, "parallelism": "single GPU"},
        "timing": f"median of {args.steps} HIP-graph replays of fwd+bwd, each after a 512 MiB cache-evicting "
                  f"write; eager launches: ms_per_step_eager",
        "ms_per_step_mean": round(statistics.fmean(res["graph_ms"]), 4),
        "ms_per_step_eager": round(ms_eager, 4),
        "pct_of_peak": round(100.0 * value / peak, 2),
        "fwd_tflops": round(fwd_flops / (fwd_ms * 1e-3) / 1e12, 2) if fwd_ms else None,
        "bwd_tflops": round(bwd_flops / (bwd_ms * 1e-3) / 1e12, 2) if bwd_ms else None,
        "kernels_ms": {k: (round(v, 4) if v else None) for k, v in kern.items()},
        "roofline": roof,
    }
    if not args.no_extras:
        out["rope"] = time_rope(binding, torch, dev, prob, args.steps, args.warmup)
        out["last"] = time_last(binding, torch, dev, prob, args.steps, args.warmup)
        out["xours"] = time_xours(binding, torch, dev, prob, args.steps, args.warmup, flush, ms)
    if not args.no_repeated:
        out["speedup_ceiling_pairs"] = round(rep_pairs / pairs, 3)
        G, P, sum_s = prob.group_sizes, prob.prefix_lens, prob.suffix_lens.sum()
        out["speedup_target"] = round(0.8 * float((G * P).sum() + sum_s) / float(P.sum() + sum_s), 3)
        del bufs
        layouts = ["repeated"] + (["padded"] if args.padded else [])
        for name in layouts:
            progress(f"building the {name} layout on the device")
            bdev, shape = baseline_layout(torch, dev, prob, padded=name == "padded")
            bbufs = alloc(binding, torch, bdev, shape)
            r = time_layout(binding, torch, bdev, bbufs, args.steps, args.warmup, flush, name, eager=False)
            rms = statistics.median(r["graph_ms"])
            progress(f"{name} layout: {rms:.3f} ms/step")
            out[f"{name}_ms_per_step"] = round(rms, 4)
            out[f"speedup_vs_{name}"] = round(rms / ms, 3)
            if name == "repeated":
                run = copy_sum_fn(torch, prob, bbufs)
                for _ in range(max(args.warmup, 1)):
                    run()
                csum = statistics.median(timed_steps(torch, run, min(args.steps, 10), flush, "prefix copy sum"))
                # reported apart: the kernels' speedup above does not include it
                out["repeated_prefix_copy_sum_ms"] = round(csum, 4)
                out["speedup_vs_repeated_with_copy_sum"] = round((rms + csum) / ms, 3)
            del bdev, bbufs
            torch.cuda.empty_cache()
        if args.padded:
            out["speedup_ceiling_pairs_padded"] = round(
                padded_pair_count(prob.prefix_lens, prob.group_sizes, prob.suffix_lens) / pairs, 3)
    del dev
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        progress("timing the CPU oracle on a sample")
        out["cpu_baseline"] = cpu_baseline(prob, args.cpu_budget)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

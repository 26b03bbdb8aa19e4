"""Seeded synthetic workloads for grouped (shared-prefix) causal attention.

This module only draws random numbers and encodes them for storage; it holds
none of the attention arithmetic. Both the CPU oracle (via the tests and the
bench's CPU leg) and the GPU path receive the arrays it produces.

Recipe (every draw is reproducible from ``seed`` alone, independent of the
number of threads used to produce it):

* lengths come from ``PCG64(SeedSequence(seed, spawn_key=(0,)))``: first the
  prefix length of every group in group order, then every suffix length,
  group-major, member order inside a group;
* tensor ``t`` (0..7 = Q_pre, K_pre, V_pre, Q_suf, K_suf, V_suf, dO_pre,
  dO_suf) is cut into chunks of ``CHUNK`` elements in row-major order, and
  chunk ``c`` is filled by ``PCG64(SeedSequence(seed, spawn_key=(1, t, c)))``
  with float32 standard normals;
* bf16 workloads round those float32 values to bfloat16 with
  round-to-nearest-even; fp32 workloads keep them;
* the "peaked" stress variant multiplies Q by 4 before rounding, which makes
  the softmax rows sharp and exercises the running-max rescale.

Shapes follow the packed varlen convention: ``*_pre`` tensors are
``[sum(P), heads, d]`` and ``*_suf`` tensors ``[sum(S), heads, d]``, groups in
order, members of a group contiguous in suffix order.
"""
from __future__ import annotations

import math
import mmap
import os
import threading
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np

CHUNK = 1 << 22
TENSOR_NAMES = ("q_pre", "k_pre", "v_pre", "q_suf", "k_suf", "v_suf", "do_pre", "do_suf")


@dataclass(frozen=True)
class Workload:
    """A workload shape: how lengths are drawn and the head geometry."""
    name: str
    n_groups: int
    group_size: int
    prefix: tuple  # ("fixed", P) or ("loguniform", lo, hi)
    suffix: tuple  # ("uniform", lo, hi), inclusive integer bounds
    h_q: int
    h_kv: int
    head_dim: int
    dtype: str  # "bf16" or "fp32"
    scale: float
    note: str = ""


WORKLOADS = {
    "tiny": Workload("tiny", 1, 4, ("fixed", 64), ("uniform", 16, 32), 2, 2, 64, "fp32", 1.0 / 8.0,
                     "1 group, G=4, P=64, S~U[16,32], H_q=H_kv=2, d=64, fp32, scale 1/sqrt(64)"),
    "single_group": Workload("single_group", 1, 8, ("fixed", 4096), ("uniform", 256, 1024), 32, 8, 128, "bf16",
                             1.0 / math.sqrt(128), "1 group, G=8, P=4096, S~U[256,1024], H_q=32, H_kv=8, d=128, bf16"),
    "long_prefix": Workload("long_prefix", 1, 16, ("fixed", 16384), ("uniform", 128, 512), 32, 8, 128, "bf16",
                            1.0 / math.sqrt(128), "1 group, G=16, P=16384, S~U[128,512], H_q=32, H_kv=8, d=128, bf16"),
    "large_group": Workload("large_group", 1, 64, ("fixed", 8192), ("uniform", 128, 2048), 40, 8, 128, "bf16",
                            1.0 / math.sqrt(128), "1 group, G=64, P=8192, S~U[128,2048], H_q=40, H_kv=8, d=128, bf16"),
    "packed_varlen": Workload("packed_varlen", 8, 16, ("loguniform", 1024, 32768), ("uniform", 64, 4096), 64, 8, 128,
                              "bf16", 1.0 / math.sqrt(128),
                              "8 groups, G=16, P~logU[1024,32768], S~U[64,4096], H_q=64, H_kv=8, d=128, bf16"),
}


@dataclass
class Problem:
    """Lengths plus host tensors of one seeded draw.

    For bf16 workloads the tensors hold bfloat16 bit patterns (uint16); for
    fp32 workloads they hold float32 values.
    """
    workload: Workload
    seed: int
    prefix_lens: np.ndarray  # int64 [n_groups]
    group_sizes: np.ndarray  # int64 [n_groups]
    suffix_lens: np.ndarray  # int64 [n_suffixes]
    tensors: dict = field(default_factory=dict)

    @property
    def h_q(self):
        return self.workload.h_q

    @property
    def h_kv(self):
        return self.workload.h_kv

    @property
    def head_dim(self):
        return self.workload.head_dim

    @property
    def scale(self):
        return self.workload.scale

    @property
    def dtype(self):
        return self.workload.dtype

    @property
    def cu_prefix(self):
        return np.concatenate([[0], np.cumsum(self.prefix_lens)]).astype(np.int64)

    @property
    def cu_suffix(self):
        return np.concatenate([[0], np.cumsum(self.suffix_lens)]).astype(np.int64)

    @property
    def total_prefix(self):
        return int(self.prefix_lens.sum())

    @property
    def total_suffix(self):
        return int(self.suffix_lens.sum())

    def as_float(self, name, dtype=np.float64):
        """Tensor ``name`` decoded to ``dtype`` (bf16 bit patterns are widened exactly)."""
        a = self.tensors[name]
        if a.dtype == np.uint16:
            a = bf16_bits_to_f32(a)
        return a.astype(dtype, copy=False)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to float32."""
    return (bits.astype(np.uint32) << 16).view(np.float32)


def _round_bf16(u: np.ndarray) -> np.ndarray:
    """float32 bit patterns (uint32) to bfloat16 bit patterns, round to nearest, ties to even."""
    return ((u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)).astype(np.uint16)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (round to nearest, ties to even); returns bit patterns."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    out = np.empty(b.shape, dtype=np.uint16)
    flat_b, flat_o = b.reshape(-1), out.reshape(-1)
    step = CHUNK

    def work(s):
        flat_o[s:s + step] = _round_bf16(flat_b[s:s + step])

    with ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(work, range(0, flat_b.size, step)))
    return out


def _threads():
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def draw_lengths(workload: Workload, seed: int):
    """Prefix lengths, group sizes and suffix lengths for one seeded draw."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=(0,))))
    ng = workload.n_groups
    if workload.prefix[0] == "fixed":
        prefix = np.full(ng, workload.prefix[1], dtype=np.int64)
    elif workload.prefix[0] == "loguniform":
        lo, hi = workload.prefix[1], workload.prefix[2]
        prefix = np.rint(np.exp(rng.uniform(math.log(lo), math.log(hi), size=ng))).astype(np.int64)
    else:
        raise ValueError(workload.prefix)
    groups = np.full(ng, workload.group_size, dtype=np.int64)
    lo, hi = workload.suffix[1], workload.suffix[2]
    suffix = rng.integers(lo, hi + 1, size=int(groups.sum()), dtype=np.int64)
    return prefix, groups, suffix


_scratch = threading.local()


def _alloc(n: int, dtype) -> np.ndarray:
    """An uninitialised 1-D array; large ones on anonymous memory advised for transparent huge pages,
    which cuts the page faults of first touch by ~500x (first touch dominated drawing the largest
    workloads)."""
    dtype = np.dtype(dtype)
    nbytes = n * dtype.itemsize
    if nbytes < (64 << 20) or not hasattr(mmap, "MADV_HUGEPAGE"):
        return np.empty(n, dtype)
    m = mmap.mmap(-1, nbytes, flags=mmap.MAP_PRIVATE | mmap.MAP_ANONYMOUS)
    m.madvise(mmap.MADV_HUGEPAGE)
    return np.frombuffer(m, dtype=dtype, count=n)


def _chunk_buffers():
    """Per-thread float32 and uint32 buffers of CHUNK elements, allocated once per thread (fresh
    arrays per chunk would make every thread page-fault on new memory, which serialises them)."""
    b = getattr(_scratch, "bufs", None)
    if b is None:
        b = (np.empty(CHUNK, np.float32), np.empty(CHUNK, np.uint32))
        _scratch.bufs = b
    return b


def normal_tensor(seed: int, tensor_index: int, shape, peaked: float = 1.0, bf16: bool = False) -> np.ndarray:
    """Float32 standard normals for tensor ``tensor_index`` (chunked, thread-count independent).

    With ``bf16`` the values are rounded to bfloat16 (nearest, ties to even) chunk by chunk as they
    are drawn and the bit patterns (uint16) are returned: the same numbers as rounding the float32
    tensor afterwards, without holding it.
    """
    n = int(np.prod(shape)) if len(shape) else 1
    out = _alloc(n, np.uint16 if bf16 else np.float32)

    def work(c):
        s = c * CHUNK
        e = min(n, s + CHUNK)
        g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=(1, tensor_index, c))))
        xb, ub = _chunk_buffers()
        x, u = xb[:e - s], ub[:e - s]
        g.standard_normal(e - s, dtype=np.float32, out=x)
        if peaked != 1.0:
            x *= np.float32(peaked)
        if bf16:
            # (bits + 0x7fff + lsb of the kept half) >> 16
            b = x.view(np.uint32)
            np.right_shift(b, np.uint32(16), out=u)
            np.bitwise_and(u, np.uint32(1), out=u)
            np.add(u, b, out=u)
            np.add(u, np.uint32(0x7FFF), out=u)
            np.right_shift(u, np.uint32(16), out=u)
            out[s:e] = u
        else:
            out[s:e] = x

    n_chunks = (n + CHUNK - 1) // CHUNK
    with ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(work, range(n_chunks)))
    return out.reshape(shape)


def make_problem(workload, seed: int = 0, lengths=None, grads: bool = True, peaked: bool = False,
                 h_q=None, h_kv=None, head_dim=None, dtype=None, scale=None) -> Problem:
    """Draw one problem.

    ``workload`` is a ``Workload`` or a name in ``WORKLOADS``. ``lengths`` may
    override the drawn lengths with ``(prefix_lens, group_sizes, suffix_lens)``;
    the head geometry, dtype and scale may be overridden the same way (used by
    edge-case tests). Tensors are always drawn from the seed as documented
    above.
    """
    if isinstance(workload, str):
        workload = WORKLOADS[workload]
    over = {k: v for k, v in dict(h_q=h_q, h_kv=h_kv, head_dim=head_dim, dtype=dtype, scale=scale).items()
            if v is not None}
    if over:
        workload = Workload(**{**workload.__dict__, **over})
    if lengths is None:
        prefix, groups, suffix = draw_lengths(workload, seed)
    else:
        prefix, groups, suffix = (np.asarray(x, dtype=np.int64) for x in lengths)
        if groups.sum() != suffix.size or prefix.size != groups.size:
            raise ValueError("inconsistent lengths")
    tp, ts = int(prefix.sum()), int(suffix.sum())
    hq, hk, d = workload.h_q, workload.h_kv, workload.head_dim
    shapes = {"q_pre": (tp, hq, d), "k_pre": (tp, hk, d), "v_pre": (tp, hk, d),
              "q_suf": (ts, hq, d), "k_suf": (ts, hk, d), "v_suf": (ts, hk, d),
              "do_pre": (tp, hq, d), "do_suf": (ts, hq, d)}
    prob = Problem(workload, seed, prefix, groups, suffix)
    for t, name in enumerate(TENSOR_NAMES):
        if name.startswith("do") and not grads:
            continue
        prob.tensors[name] = normal_tensor(seed, t, shapes[name], peaked=4.0 if (peaked and name.startswith("q")) else 1.0,
                                           bf16=workload.dtype == "bf16")
    return prob


def xours_order(prob: Problem) -> np.ndarray:
    """Row order of the single-buffer layout of Eq. (2): group after group, the group's prefix rows and then
    its members' response rows. Entry i is the packed row (prefix rows 0..total_prefix-1, then response rows
    from total_prefix on) that goes to row i of the single buffer."""
    cu_p, cu_s, tp = prob.cu_prefix, prob.cu_suffix, prob.total_prefix
    order, m = [], 0
    for g, gs in enumerate(prob.group_sizes):
        order.append(np.arange(cu_p[g], cu_p[g + 1]))
        order.append(tp + np.arange(cu_s[m], cu_s[m + int(gs)]))
        m += int(gs)
    return np.concatenate(order).astype(np.int64) if order else np.zeros(0, np.int64)


def repeated_layout(prob: Problem) -> Problem:
    """The repeated-prefix layout of ``prob``: every member gets its own copy of its group's prefix.

    The result has one group per member (``group_sizes`` all 1), the member's
    prefix rows copied in front; ``do_pre`` of a group is handed whole to its
    first member and zero to the others, so the summed prefix gradients of the
    copies equal the grouped ones. Groups with no members keep their prefix as
    a group of size 0.
    """
    cu_p, cu_s = prob.cu_prefix, prob.cu_suffix
    pre_idx, suf_idx, prefix, groups, suffix, first = [], [], [], [], [], []
    m = 0
    for g, (p, gs) in enumerate(zip(prob.prefix_lens, prob.group_sizes)):
        rows = np.arange(cu_p[g], cu_p[g + 1])
        if gs == 0:
            pre_idx.append(rows); prefix.append(p); groups.append(0); first.append(True)
        for i in range(gs):
            pre_idx.append(rows); prefix.append(p); groups.append(1); first.append(i == 0)
            suf_idx.append(np.arange(cu_s[m], cu_s[m + 1])); suffix.append(prob.suffix_lens[m]); m += 1
    pre_idx = np.concatenate(pre_idx) if pre_idx else np.zeros(0, np.int64)
    suf_idx = np.concatenate(suf_idx) if suf_idx else np.zeros(0, np.int64)
    rep = Problem(prob.workload, prob.seed, np.array(prefix, np.int64), np.array(groups, np.int64),
                  np.array(suffix, np.int64))
    keep = np.concatenate([np.full(p, f) for p, f in zip(prefix, first)]) if prefix else np.zeros(0, bool)
    for name, a in prob.tensors.items():
        if name.endswith("_pre"):
            r = a[pre_idx]
            if name == "do_pre":
                r = r.copy()
                r[~keep] = 0
            rep.tensors[name] = r
        else:
            rep.tensors[name] = a[suf_idx]
    return rep

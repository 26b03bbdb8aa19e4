"""GPU parity of the grouped-position rotary embedding (pg_rope, pg_grouped_positions) against the oracle.

Positions are integers and compared exactly. Rotated values are compared
element by element: fp32 mode within 1e-5 absolute (the rotation of N(0, 1)
inputs in fp32 arithmetic with cos / sin rounded once to fp32); bf16 mode
within half a bf16 unit in the last place of the exact result (2^-8 of its
magnitude, the single rounding of the fp32 result) plus 1e-6.
"""
import numpy as np
import pytest

from oracle import grouped_oracle, grouped_positions, rope
from paper_2506_05433_amd.inputs import make_problem
from tests._parity import check, host_view, to_host

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

FP32_ABS = 1e-5


def _dev():
    from paper_2506_05433_amd import binding
    assert torch.cuda.is_available(), "GPU test needs a GPU"
    binding.lib()
    return binding


def _compare(name, got, ref, dtype):
    got = np.asarray(got, np.float64)
    assert got.shape == ref.shape, (name, got.shape, ref.shape)
    err = np.abs(got - ref)
    if dtype == "fp32":
        bound = np.full_like(ref, FP32_ABS)
    else:
        bound = 2.0 ** -8 * np.abs(ref) + 1e-6
    worst = float((err - bound).max()) if err.size else 0.0
    print(f"{name}: max_abs={float(err.max()) if err.size else 0:.3e} worst excess={worst:.3e}", flush=True)
    assert worst <= 0.0, f"{name}: error above bound by {worst:.3e}"


def _rope_case(prob, base=10000.0, rotary_dim=None, inverse=False, interleaved=False, in_place=False):
    binding = _dev()
    print(f"[rope] {prob.dtype} P={list(prob.prefix_lens)[:4]} G={list(prob.group_sizes)[:4]} "
          f"h={prob.h_q}/{prob.h_kv} d={prob.head_dim} rot={rotary_dim} inv={inverse} inter={interleaved} "
          f"in_place={in_place}", flush=True)
    dev = binding.to_device(prob, "cuda")
    names = ("q_pre", "q_suf", "k_pre", "k_suf")
    ins = tuple(dev[n] for n in names)
    keep = tuple(t.clone() for t in ins)
    out = ins if in_place else None
    got = binding.rope(*ins, dev["cu_prefix"], dev["cu_suffix"], dev["group_sizes"], base=base,
                       rotary_dim=rotary_dim, inverse=inverse, interleaved=interleaved, out=out)
    torch.cuda.synchronize()
    if not in_place:
        for a, b in zip(ins, keep):
            assert torch.equal(a, b), "pg_rope wrote to its input"
    pos_pre, pos_suf = grouped_positions(prob.prefix_lens, prob.group_sizes, prob.suffix_lens)
    t = host_view(prob)
    for n, g in zip(names, got):
        pos = pos_pre if n.endswith("_pre") else pos_suf
        ref = rope(np.asarray(t[n], np.float64), pos, base, rotary_dim, interleaved=interleaved, inverse=inverse)
        _compare(n, to_host(g), ref, prob.dtype)
        if rotary_dim is not None and rotary_dim < prob.head_dim:
            tail = to_host(g)[..., rotary_dim:]
            assert np.array_equal(tail, np.asarray(t[n], np.float32)[..., rotary_dim:]), "pass-through changed"


def test_positions_match_oracle():
    binding = _dev()
    for lengths in (((300,), (5,), (130, 1, 64, 200, 97)),
                    ((3, 0, 200, 1), (2, 1, 0, 3), (5, 0, 7, 1, 1, 130)),
                    ((0,), (1,), (5,)),
                    ((7,), (0,), ()),
                    ((4096, 100, 7), (8, 1, 2), (256, 1024, 999, 3, 512, 640, 700, 1, 17, 2, 30))):
        prob = make_problem("tiny", seed=1, lengths=lengths)
        dev = binding.to_device(prob, "cuda")
        got = binding.grouped_positions(prob.total_prefix, prob.total_suffix, dev["cu_prefix"], dev["cu_suffix"],
                                        dev["group_sizes"])
        ref = grouped_positions(prob.prefix_lens, prob.group_sizes, prob.suffix_lens)
        for g, r in zip(got, ref):
            assert np.array_equal(g.cpu().numpy(), r), lengths


@pytest.mark.parametrize("inverse", [False, True])
@pytest.mark.parametrize("interleaved", [False, True])
def test_rope_fp32_tiny(inverse, interleaved):
    _rope_case(make_problem("tiny", seed=0), inverse=inverse, interleaved=interleaved)


@pytest.mark.parametrize("rot,dt", [(64, "bf16"), (32, "fp32"), (16, "bf16")])
def test_rope_partial_rotary(rot, dt):
    prob = make_problem("single_group", seed=11, lengths=((300, 0), (3, 1), (200, 5, 1, 64)), h_q=4, h_kv=2,
                        head_dim=128 if rot > 16 else 64, dtype=dt)
    _rope_case(prob, base=500000.0, rotary_dim=rot)


def test_rope_edge_groups_in_place():
    prob = make_problem("single_group", seed=12, lengths=((3, 0, 200, 1), (2, 1, 0, 3), (5, 0, 7, 1, 1, 130)),
                        h_q=8, h_kv=1, head_dim=128)
    _rope_case(prob, in_place=True)


def test_rope_bf16_single_group_full():
    """The bench workload at full size (32 query and 8 key heads, positions up to 5120), every element."""
    _rope_case(make_problem("single_group", seed=0))


def test_rope_long_positions_interleaved():
    """Positions past 16000 (long_prefix): the angle is computed in double precision."""
    prob = make_problem("long_prefix", seed=0, h_q=4, h_kv=2)
    _rope_case(prob, base=1000000.0, interleaved=True)


def test_rope_then_attention_matches_oracle():
    """The step before the kernel: rope on the GPU then the grouped attention, against the oracle's rope and
    attention, forward and backward (the gradients of the unrotated q, k come from the inverse rotation)."""
    binding = _dev()
    prob = make_problem("single_group", seed=13, lengths=((300, 40), (3, 2), (130, 1, 64, 200, 97)), h_q=4,
                        h_kv=2, head_dim=128, dtype="fp32", scale=1.0 / np.sqrt(128))
    dev = binding.to_device(prob, "cuda")
    rq_pre, rq_suf, rk_pre, rk_suf = binding.rope(dev["q_pre"], dev["q_suf"], dev["k_pre"], dev["k_suf"],
                                                  dev["cu_prefix"], dev["cu_suffix"], dev["group_sizes"])
    args = (dev["cu_prefix"], dev["cu_suffix"], dev["group_sizes"], dev["scale"])
    f = binding.fwd(rq_pre, rk_pre, dev["v_pre"], rq_suf, rk_suf, dev["v_suf"], *args)
    dq_pre, dk_pre, dv_pre, dq_suf, dk_suf, dv_suf = binding.bwd(
        rq_pre, rk_pre, dev["v_pre"], rq_suf, rk_suf, dev["v_suf"], *f, dev["do_pre"], dev["do_suf"], *args)
    gq_pre, gq_suf, gk_pre, gk_suf = binding.rope(dq_pre, dq_suf, dk_pre, dk_suf, dev["cu_prefix"],
                                                  dev["cu_suffix"], dev["group_sizes"], inverse=True)
    torch.cuda.synchronize()
    # oracle: rotate, attend, and map the rotated-q/k gradients back with the rotation's transpose
    t = {k: np.asarray(v, np.float64) for k, v in host_view(prob).items()}
    pos_pre, pos_suf = grouped_positions(prob.prefix_lens, prob.group_sizes, prob.suffix_lens)
    for n in ("q_pre", "k_pre"):
        t[n] = rope(t[n], pos_pre, 10000.0)
    for n in ("q_suf", "k_suf"):
        t[n] = rope(t[n], pos_suf, 10000.0)
    ref = grouped_oracle(prob.prefix_lens, prob.group_sizes, prob.suffix_lens, t, prob.scale, grads=True)
    check("o_pre", to_host(f[0]), ref["o_pre"], "fp32")
    check("o_suf", to_host(f[1]), ref["o_suf"], "fp32")
    check("dv_pre", to_host(dv_pre), ref["dv_pre"], "fp32")
    for name, got, pos in (("dq_pre", gq_pre, pos_pre), ("dq_suf", gq_suf, pos_suf),
                           ("dk_pre", gk_pre, pos_pre), ("dk_suf", gk_suf, pos_suf)):
        check(name, to_host(got), rope(ref[name], pos, 10000.0, inverse=True), "fp32")

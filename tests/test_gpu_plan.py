"""The one-block planner and the multi-kernel planner give the same plan.

Problems whose tile lists fit one block of the planner are planned by a single fused kernel; larger
ones by the sequence of planner kernels. PG_PLAN_MULTI=1 forces the sequence, so running the same
calls both ways must give bitwise-identical outputs and gradients (split and single-buffer layouts,
with the dK/dV prefix walks cut into several pieces and not), and the planner's verdict on
inconsistent grouping arrays must be the same.
"""
import os

import numpy as np
import pytest

from paper_2506_05433_amd.inputs import make_problem, xours_order
from tests._parity import GRADS, OUTS, to_host

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

_rng = np.random.default_rng(12)
_G = _rng.integers(0, 3, 400)
CASES = [
    # 400 small groups: still one block's worth of tiles, several passes of nothing else
    (tuple(_rng.integers(0, 70, 400)), tuple(_G), tuple(_rng.integers(0, 40, int(_G.sum()))), 2, 1, 64, "fp32"),
    ((257, 0, 40), (3, 2, 0), (129, 128, 1, 300, 0), 4, 2, 64, "bf16"),
    ((900,), (6,), (100, 300, 1, 250, 64, 129), 8, 2, 128, "bf16"),
    ((64,), (4,), (16, 31, 20, 32), 2, 2, 64, "fp32"),
    ((0, 70, 5), (2, 0, 3), (9, 0, 33, 1, 77), 4, 1, 128, "fp32"),
]


def _both(fn):
    """fn() with the fused planner, then with the multi-kernel planner."""
    old = os.environ.pop("PG_PLAN_MULTI", None)
    try:
        a = fn()
        os.environ["PG_PLAN_MULTI"] = "1"
        b = fn()
    finally:
        os.environ.pop("PG_PLAN_MULTI", None)
        if old is not None:
            os.environ["PG_PLAN_MULTI"] = old
    return a, b


@pytest.mark.parametrize("case", range(len(CASES)))
def test_fused_planner_matches_kernel_sequence(case):
    from paper_2506_05433_amd import binding
    assert torch.cuda.is_available(), "GPU test needs a GPU"
    prefix, groups, suffix, hq, hkv, d, dt = CASES[case]
    lengths = (prefix, groups, suffix)
    prob = make_problem("single_group", seed=700 + case, lengths=lengths, h_q=hq, h_kv=hkv, head_dim=d, dtype=dt,
                        scale=1.0 / np.sqrt(d))
    print(f"[plan] case {case}: {lengths} h={hq}/{hkv} d={d} {dt}", flush=True)
    dev = binding.to_device(prob, "cuda")
    order = torch.as_tensor(xours_order(prob), device="cuda")
    x = {n: torch.cat([dev[n + "_pre"], dev[n + "_suf"]])[order] for n in ("q", "k", "v", "do")}
    grp = (dev["cu_prefix"], dev["cu_suffix"], dev["group_sizes"], prob.total_prefix, dev["scale"])

    def run():
        f = binding.run_fwd(dev)
        g = binding.run_bwd(dev, f)
        o, lse = binding.fwd_xours(x["q"], x["k"], x["v"], *grp)
        xg = binding.bwd_xours(x["q"], x["k"], x["v"], o, lse, x["do"], *grp)
        torch.cuda.synchronize()
        out = dict(zip(OUTS, f))
        out.update(zip(GRADS, g))
        out.update(x_o=o, x_lse=lse, x_dq=xg[0], x_dk=xg[1], x_dv=xg[2])
        return {k: to_host(v) for k, v in out.items()}

    fused, multi = _both(run)
    for k in fused:
        assert np.array_equal(fused[k], multi[k]), f"{k}: the two planners gave different results"


def test_both_planners_reject_inconsistent_arrays():
    """Decreasing response offsets: no work is done, and PG_DEBUG_VALIDATE=1 reports PG_EINVAL, either way."""
    from paper_2506_05433_amd import binding
    prob = make_problem("single_group", seed=710, lengths=((40,), (2,), (5, 7)), h_q=2, h_kv=1, head_dim=64,
                        dtype="fp32")
    dev = binding.to_device(prob, "cuda")
    dev["cu_suffix"] = torch.tensor([0, 9, 3], dtype=torch.int32, device="cuda")  # not nondecreasing

    def run():
        o_pre = torch.full_like(dev["q_pre"], 7.0)
        o_suf = torch.full_like(dev["q_suf"], 7.0)
        lp = torch.zeros(2, 40, device="cuda")
        ls = torch.zeros(2, 12, device="cuda")
        binding.fwd(dev["q_pre"], dev["k_pre"], dev["v_pre"], dev["q_suf"], dev["k_suf"], dev["v_suf"],
                    dev["cu_prefix"], dev["cu_suffix"], dev["group_sizes"], dev["scale"], out=(o_pre, o_suf, lp, ls))
        torch.cuda.synchronize()
        untouched = bool((o_pre == 7.0).all()) and bool((o_suf == 7.0).all())
        os.environ["PG_DEBUG_VALIDATE"] = "1"
        try:
            with pytest.raises(binding.PgError) as e:
                binding.run_fwd(dev)
        finally:
            os.environ.pop("PG_DEBUG_VALIDATE", None)
        return untouched, e.value.status

    assert _both(run) == ((True, 1), (True, 1))

"""Seeded random groupings on the GPU against the oracle: every entry point on the same problem.

Each case draws the number of groups, their prefix lengths (0 allowed), member counts (0 allowed) and
response lengths (0 allowed), a GQA ratio, head_dim and dtype, then checks the split-layout forward and
backward element by element, the single-buffer calls bit for bit against the split ones, the final-token
forward against the oracle's per-row evaluation, and the rotary embedding against its oracle.
"""
import numpy as np
import pytest

from oracle import grouped_oracle, grouped_positions, rope
from paper_2506_05433_amd.inputs import make_problem, xours_order
from tests._parity import GRADS, OUTS, check, host_view, to_host
from tests.test_gpu_last import _oracle_last

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

N_CASES = 12


def _draw(case):
    rng = np.random.default_rng(9000 + case)
    ng = int(rng.integers(1, 5))
    prefix = [int(rng.choice([0, rng.integers(1, 64), rng.integers(64, 700)])) for _ in range(ng)]
    groups = [int(rng.integers(0, 6)) for _ in range(ng)]
    if sum(groups) == 0:
        groups[0] = 1
    suffix = [int(rng.choice([0, rng.integers(1, 40), rng.integers(40, 300)])) for _ in range(sum(groups))]
    ratio = int(rng.choice([1, 2, 4, 5, 8]))
    h_kv = int(rng.integers(1, 3))
    d = int(rng.choice([64, 128]))
    dtype = "fp32" if case % 4 == 3 else "bf16"
    return (tuple(prefix), tuple(groups), tuple(suffix)), ratio * h_kv, h_kv, d, dtype


@pytest.mark.parametrize("case", range(N_CASES))
def test_random_grouping(case):
    from paper_2506_05433_amd import binding
    assert torch.cuda.is_available(), "GPU test needs a GPU"
    lengths, hq, hkv, d, dt = _draw(case)
    print(f"[random {case}] lengths={lengths} h={hq}/{hkv} d={d} {dt}", flush=True)
    prob = make_problem("single_group", seed=9100 + case, lengths=lengths, h_q=hq, h_kv=hkv, head_dim=d, dtype=dt,
                        scale=1.0 / np.sqrt(d))
    dev = binding.to_device(prob, "cuda")
    f = binding.run_fwd(dev)
    g = binding.run_bwd(dev, f)
    names = ("q_pre", "k_pre", "v_pre", "q_suf", "k_suf", "v_suf")
    grp = (dev["cu_prefix"], dev["cu_suffix"], dev["group_sizes"])
    o_last, lse_last = binding.fwd_last(*[dev[n] for n in names], *grp, dev["scale"])
    order = torch.as_tensor(xours_order(prob), device="cuda")
    x = {n: torch.cat([dev[n + "_pre"], dev[n + "_suf"]])[order] for n in ("q", "k", "v", "do")}
    xo, xlse = binding.fwd_xours(x["q"], x["k"], x["v"], *grp, prob.total_prefix, dev["scale"])
    xdq, xdk, xdv = binding.bwd_xours(x["q"], x["k"], x["v"], xo, xlse, x["do"], *grp, prob.total_prefix,
                                      dev["scale"])
    rq = binding.rope(dev["q_pre"], dev["q_suf"], dev["k_pre"], dev["k_suf"], *grp, base=10000.0)
    torch.cuda.synchronize()

    ref = grouped_oracle(prob.prefix_lens, prob.group_sizes, prob.suffix_lens, host_view(prob), prob.scale,
                         grads=True)
    for name, t in zip(OUTS + GRADS, list(f) + list(g)):
        check(name, to_host(t), ref[name], dt)
    # single-buffer layout: bitwise the split results, reordered
    for name, xt, pre, suf in (("o", xo, f[0], f[1]), ("dq", xdq, g[0], g[3]), ("dk", xdk, g[1], g[4]),
                               ("dv", xdv, g[2], g[5])):
        assert torch.equal(xt, torch.cat([pre, suf])[order]), f"xours {name}"
    assert torch.equal(xlse, torch.cat([f[2], f[3]], dim=1)[:, order]), "xours lse"
    # final-token forward
    ro, rl = _oracle_last(prob, list(range(hq)))
    finite = np.isfinite(rl)
    check("o_last", to_host(o_last), ro, dt)
    assert np.array_equal(np.isfinite(to_host(lse_last)), finite)
    check("lse_last", np.where(finite, to_host(lse_last), 0), np.where(finite, rl, 0), dt)
    # rotary embedding (bf16: half an ulp of the exact result; fp32: 1e-5)
    pos_pre, pos_suf = grouped_positions(prob.prefix_lens, prob.group_sizes, prob.suffix_lens)
    t = host_view(prob)
    for name, got, pos in zip(("q_pre", "q_suf", "k_pre", "k_suf"), rq, (pos_pre, pos_suf, pos_pre, pos_suf)):
        exact = rope(np.asarray(t[name], np.float64), pos, 10000.0)
        err = np.abs(to_host(got) - exact)
        bound = 1e-5 if dt == "fp32" else 2.0 ** -8 * np.abs(exact) + 1e-6
        assert np.all(err <= bound), f"rope {name}: {float((err - bound).max()):.3e} above bound"

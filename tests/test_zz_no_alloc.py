"""pg_attn_fwd_noalloc (the forward without a workspace, for callers that cannot allocate) against
pg_attn_fwd on the same inputs: bitwise equal outputs on two calls in a row, the second smaller than the
first (the scratch array keeps the first call's plan, which the second must not read)."""
import numpy as np
import pytest

from paper_2506_05433_amd.inputs import make_problem
from tests._parity import OUTS, check, host_view, to_host

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _outputs_like(dev, prob):
    return (torch.full_like(dev["q_pre"], 3.0), torch.full_like(dev["q_suf"], 3.0),
            torch.full((prob.h_q, prob.total_prefix), 3.0, device="cuda"),
            torch.full((prob.h_q, prob.total_suffix), 3.0, device="cuda"))


def _both(prob):
    from paper_2506_05433_amd import binding
    assert torch.cuda.is_available(), "GPU test needs a GPU"
    print(f"[no_alloc] P={list(prob.prefix_lens)} G={list(prob.group_sizes)} S={list(prob.suffix_lens)} "
          f"hq={prob.h_q} hkv={prob.h_kv} d={prob.head_dim} {prob.dtype}", flush=True)
    dev = binding.to_device(prob, "cuda")
    ref = binding.run_fwd(dev)
    got = binding.fwd_noalloc(dev["q_pre"], dev["k_pre"], dev["v_pre"], dev["q_suf"], dev["k_suf"], dev["v_suf"],
                              dev["cu_prefix"], dev["cu_suffix"], dev["group_sizes"], dev["scale"],
                              out=_outputs_like(dev, prob))
    torch.cuda.synchronize()
    return [to_host(t) for t in got], [to_host(t) for t in ref]


def test_noalloc_forward_equals_workspace_forward_twice_shrinking():
    big = make_problem("single_group", seed=21, lengths=((700, 130), (4, 2), (300, 90, 211, 5, 64, 129)), h_q=8,
                       h_kv=2, head_dim=128)
    small = make_problem("single_group", seed=22, lengths=((100,), (2,), (30, 7)), h_q=4, h_kv=1, head_dim=64)
    for prob in (big, small):
        got, ref = _both(prob)
        for name, g, r in zip(OUTS, got, ref):
            assert np.array_equal(g, r), name
    # and the second (smaller) call against the oracle
    from oracle import grouped_oracle
    o = grouped_oracle(small.prefix_lens, small.group_sizes, small.suffix_lens, host_view(small), small.scale,
                       grads=False)
    for name, g in zip(OUTS, got):
        check(name, g, o[name], small.dtype)


def test_noalloc_plan_status_reports_inconsistent_grouping():
    """With inconsistent grouping arrays the allocation-free forward does no work, and pg_plan_status reads
    that verdict from the scratch array; a consistent call after it clears it."""
    from paper_2506_05433_amd import binding
    prob = make_problem("single_group", seed=23, lengths=((64,), (2,), (10, 20)), h_q=2, h_kv=1, head_dim=64)
    dev = binding.to_device(prob, "cuda")
    out = _outputs_like(dev, prob)
    bad = torch.tensor([0, 25, 20], dtype=torch.int32, device="cuda")  # not nondecreasing
    args = (dev["q_pre"], dev["k_pre"], dev["v_pre"], dev["q_suf"], dev["k_suf"], dev["v_suf"], dev["cu_prefix"])
    binding.fwd_noalloc(*args, bad, dev["group_sizes"], dev["scale"], out=out)
    with pytest.raises(binding.PgError) as e:
        binding.plan_status()
    assert e.value.status == 1
    assert bool((out[0] == 3.0).all()) and bool((out[1] == 3.0).all())
    binding.fwd_noalloc(*args, dev["cu_suffix"], dev["group_sizes"], dev["scale"], out=out)
    binding.plan_status()
    ref = binding.run_fwd(dev)
    torch.cuda.synchronize()
    for g, r in zip(out, ref):
        assert torch.equal(g, r)

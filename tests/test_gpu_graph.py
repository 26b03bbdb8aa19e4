"""The attention calls under HIP graph capture (torch.cuda.graphs): the library launches only on the caller's
stream and records no memset, so a captured forward + backward can be replayed. Each replay, with eager work
of the program in between, must reproduce the eager results bit for bit."""
import numpy as np
import pytest

from paper_2506_05433_amd.inputs import make_problem

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def test_graph_replay_matches_eager():
    from paper_2506_05433_amd import binding
    assert torch.cuda.is_available(), "GPU test needs a GPU"
    prob = make_problem("single_group", seed=21, lengths=((300, 0, 40), (3, 1, 2), (130, 1, 64, 0, 97, 5)), h_q=8,
                        h_kv=2, head_dim=128)
    print("[graph] capture fwd+bwd and replay", flush=True)
    dev = binding.to_device(prob, "cuda")
    names = ("q_pre", "k_pre", "v_pre", "q_suf", "k_suf", "v_suf")
    args = (dev["cu_prefix"], dev["cu_suffix"], dev["group_sizes"], dev["scale"])
    ng, ns = len(prob.prefix_lens), len(prob.suffix_lens)
    sizes = (ng, ns, prob.total_prefix, prob.total_suffix, prob.h_q, prob.h_kv, prob.head_dim)
    ws_f = torch.empty(binding.workspace_bytes("fwd", *sizes), device="cuda", dtype=torch.uint8)
    ws_b = torch.empty(binding.workspace_bytes("bwd", *sizes), device="cuda", dtype=torch.uint8)
    fo = (torch.empty_like(dev["q_pre"]), torch.empty_like(dev["q_suf"]),
          torch.empty((prob.h_q, prob.total_prefix), device="cuda"), torch.empty((prob.h_q, prob.total_suffix),
                                                                                device="cuda"))
    bo = tuple(torch.empty_like(dev[n]) for n in ("q_pre", "k_pre", "v_pre", "q_suf", "k_suf", "v_suf"))

    def step():
        binding.fwd(*[dev[n] for n in names], *args, out=fo, workspace=ws_f)
        binding.bwd(*[dev[n] for n in names], *fo, dev["do_pre"], dev["do_suf"], *args, out=bo, workspace=ws_b)

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()  # warm up on the side stream before capture
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    eager = [t.clone() for t in fo + bo]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    for rep in range(3):
        for t in fo + bo:
            t.fill_(float("nan"))       # eager work between replays; the replay must overwrite it all
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(zip(fo + bo, eager)):
            assert torch.equal(a, b), f"replay {rep}: output {i} differs from the eager result"
    print("[graph] 3 replays bitwise equal to eager", flush=True)

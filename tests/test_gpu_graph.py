"""HIP-graph replay of the two entry points: a captured step (marginals on the capture
stream, Viterbi on a side stream, forked and joined with events) must give bitwise the
eager results on every replay, with unrelated eager work and synchronisations between the
replays.  The library's kernels record no memset or allocation, so the captured graph holds
kernel and event nodes only."""
import numpy as np
import pytest

from paper_2002_00876_amd import workloads as W
from gpu_util import say

pytestmark = pytest.mark.gpu


def _outputs(dev, B, N, C):
    import torch
    return (torch.empty(B, dtype=torch.float32, device=dev),
            torch.empty((B, N - 1, C, C), dtype=torch.float32, device=dev),
            torch.empty((B, N), dtype=torch.int32, device=dev),
            torch.empty(B, dtype=torch.float32, device=dev))


@pytest.mark.parametrize("case", ["paper", "tree_c40", "chunk_c64", "bf16_c128"])
def test_graph_replay_matches_eager(case, monkeypatch):
    import torch
    from paper_2002_00876_amd import binding
    if case == "paper":
        pot_h, lens_h = W.generate("paper")
    elif case == "tree_c40":
        monkeypatch.setenv("TS_PATH", "tree")
        pot_h, lens_h = W.random_case(11, 3, 37, 40)
    elif case == "chunk_c64":      # the chunk path (C <= 64, long chains)
        pot_h, lens_h = W.random_case(13, 4, 300, 64, lengths=[300, 257, 64, 2])
    else:                          # the tree with the bf16-split 128-wide tiles
        pot_h, lens_h = W.random_case(14, 4, 257, 128, lengths=[257, 200, 131, 64])
    say(f"graph replay case {case}: shape {pot_h.shape}")
    dev = torch.device("cuda:0")
    pot = torch.from_numpy(pot_h).to(dev)
    lens = torch.from_numpy(lens_h).to(dev)
    B, E, C, _ = pot.shape
    N = E + 1
    ws_m = binding._workspace(binding.OP_MARGINALS, B, N, C, dev)[0]
    ws_v = binding._workspace(binding.OP_VITERBI, B, N, C, dev)[0]

    ref = _outputs(dev, B, N, C)
    binding.marginals(pot, lens, out=(ref[0], ref[1]), ws=ws_m)
    binding.viterbi(pot, lens, out=(ref[2], ref[3]), ws=ws_v)
    torch.cuda.synchronize()
    ref = [t.cpu() for t in ref]

    out = _outputs(dev, B, N, C)
    side = torch.cuda.Stream(device=dev)
    cap = torch.cuda.Stream(device=dev)
    graph = torch.cuda.CUDAGraph()
    cap.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(cap):
        with torch.cuda.graph(graph, stream=cap):
            s = torch.cuda.current_stream(dev)
            fork = torch.cuda.Event()
            fork.record(s)
            side.wait_event(fork)
            binding.marginals(pot, lens, out=(out[0], out[1]), ws=ws_m)
            with torch.cuda.stream(side):
                binding.viterbi(pot, lens, out=(out[2], out[3]), ws=ws_v)
            join = torch.cuda.Event()
            join.record(side)
            s.wait_event(join)
    torch.cuda.current_stream(dev).wait_stream(cap)
    torch.cuda.synchronize()

    other_h, other_l = W.random_case(12, B, N, C)
    other = torch.from_numpy(other_h).to(dev)
    other_len = torch.from_numpy(other_l).to(dev)
    for rep in range(4):
        for t in out:
            t.fill_(-7)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for got, want, name in zip(out, ref, ("logZ", "marginals", "path", "score")):
            assert torch.equal(got.cpu(), want), f"replay {rep}: {name} differs from eager"
        # unrelated eager work on the same buffers' workspaces between replays
        binding.marginals(other, other_len, ws=ws_m)
        binding.viterbi(other, other_len, ws=ws_v)
        torch.cuda.synchronize()
    say(f"graph replay case {case}: 4 replays bitwise equal to eager")


@pytest.mark.parametrize("case", ["paper", "tree_c40", "bf16_c128"])
def test_graph_replay_of_the_combined_call(case, monkeypatch):
    """The combined call captured as it stands: on the multi-launch tree it forks its Viterbi
    half onto the library's side stream and joins it back, which the capture must follow."""
    import torch
    from paper_2002_00876_amd import binding
    if case == "paper":
        pot_h, lens_h = W.generate("paper")
    elif case == "tree_c40":
        monkeypatch.setenv("TS_PATH", "tree")
        pot_h, lens_h = W.random_case(13, 3, 37, 40)
    else:
        pot_h, lens_h = W.random_case(15, 4, 257, 128, lengths=[257, 190, 77, 3])
    say(f"combined-call graph case {case}: shape {pot_h.shape}")
    dev = torch.device("cuda:0")
    pot = torch.from_numpy(pot_h).to(dev)
    lens = torch.from_numpy(lens_h).to(dev)
    B, E, C, _ = pot.shape
    N = E + 1
    ws = binding._workspace(binding.OP_MARGINALS_VITERBI, B, N, C, dev)[0]
    ref = _outputs(dev, B, N, C)
    binding.marginals_viterbi(pot, lens, out=ref, ws=ws)
    torch.cuda.synchronize()
    ref = [t.cpu() for t in ref]

    out = _outputs(dev, B, N, C)
    cap = torch.cuda.Stream(device=dev)
    graph = torch.cuda.CUDAGraph()
    cap.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(cap):
        with torch.cuda.graph(graph, stream=cap):
            binding.marginals_viterbi(pot, lens, out=out, ws=ws)
    torch.cuda.current_stream(dev).wait_stream(cap)
    torch.cuda.synchronize()

    other_h, other_l = W.random_case(14, B, N, C)
    other = torch.from_numpy(other_h).to(dev)
    other_len = torch.from_numpy(other_l).to(dev)
    for rep in range(4):
        for t in out:
            t.fill_(-7)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for got, want, name in zip(out, ref, ("logZ", "marginals", "path", "score")):
            assert torch.equal(got.cpu(), want), f"replay {rep}: {name} differs from eager"
        binding.marginals_viterbi(other, other_len, ws=ws)   # eager work on the same workspace
        torch.cuda.synchronize()
    say(f"combined-call graph case {case}: 4 replays bitwise equal to eager")

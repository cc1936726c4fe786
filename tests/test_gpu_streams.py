"""Concurrent calls: the boundary allows calls with distinct workspaces to run at the same
time on different streams.  Two problems on two paths (the bf16-tile tree and the chunk
path) are enqueued on two streams, interleaved and without synchronisation between them,
several times over; every output must equal bitwise that of the same call run alone."""
import pytest

from paper_2002_00876_amd import workloads as W
from gpu_util import say

pytestmark = pytest.mark.gpu


def _problem(dev, seed, B, N, C, lens):
    import torch
    from paper_2002_00876_amd import binding
    pot_h, lens_h = W.random_case(seed, B, N, C, lengths=lens)
    pot = torch.from_numpy(pot_h).to(dev)
    tl = torch.from_numpy(lens_h).to(dev)
    ws = {op: binding._workspace(op, B, N, C, dev)[0]
          for op in (binding.OP_MARGINALS, binding.OP_VITERBI, binding.OP_MARGINALS_VITERBI)}
    return pot, tl, ws


def _outputs(dev, pot):
    import torch
    B, E, C, _ = pot.shape
    return (torch.empty(B, dtype=torch.float32, device=dev), torch.empty_like(pot),
            torch.empty((B, E + 1), dtype=torch.int32, device=dev),
            torch.empty(B, dtype=torch.float32, device=dev))


def _run(binding, prob, out, combined):
    pot, tl, ws = prob
    if combined:
        binding.marginals_viterbi(pot, tl, out=out, ws=ws[binding.OP_MARGINALS_VITERBI])
    else:
        binding.marginals(pot, tl, out=(out[0], out[1]), ws=ws[binding.OP_MARGINALS])
        binding.viterbi(pot, tl, out=(out[2], out[3]), ws=ws[binding.OP_VITERBI])


@pytest.mark.parametrize("combined", [False, True])
def test_two_streams_match_single_calls(combined):
    import torch
    from paper_2002_00876_amd import binding
    dev = torch.device("cuda:0")
    probs = [_problem(dev, 21, 4, 257, 128, [257, 200, 131, 64]),
             _problem(dev, 22, 6, 300, 64, [300, 299, 150, 64, 5, 1])]
    refs = []
    for prob in probs:
        out = _outputs(dev, prob[0])
        _run(binding, prob, out, combined)
        torch.cuda.synchronize()
        refs.append([t.cpu() for t in out])
    streams = [torch.cuda.Stream(device=dev), torch.cuda.Stream(device=dev)]
    outs = [_outputs(dev, p[0]) for p in probs]
    for rep in range(3):
        for o in outs:
            for t in o:
                t.fill_(-7)
        torch.cuda.synchronize()
        for s in streams:
            s.wait_stream(torch.cuda.current_stream(dev))
        for k in range(2):          # interleaved: both problems in flight at once
            for prob, out, s in zip(probs, outs, streams):
                with torch.cuda.stream(s):
                    _run(binding, prob, out, combined)
        torch.cuda.synchronize()
        for i, (o, ref) in enumerate(zip(outs, refs)):
            for got, want, name in zip(o, ref, ("logZ", "marginals", "path", "score")):
                assert torch.equal(got.cpu(), want), f"rep {rep}, problem {i}: {name} differs"
    say(f"two streams ({'combined call' if combined else 'separate calls'}): 3 rounds bitwise "
        "equal to the single calls")

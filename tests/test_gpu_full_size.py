"""Parity at the full sizes of the larger workloads, in the launch configuration the
benchmark uses: log Z of every sequence, Viterbi path and score of every sequence, and
marginals on sampled edges computed one sequence at a time by the oracle, plus the
sum-to-one and padding properties on every edge."""
import numpy as np
import pytest

from gpu_util import MARG_ATOL, check_logz, say
from paper_2002_00876_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["mid", "long", "hmm"])
def test_full_size(name):
    import torch

    import oracle
    from paper_2002_00876_amd import binding

    say(f"{name}: generating")
    pot, lens = W.generate(name)
    B, E, C, _ = pot.shape
    tp = torch.from_numpy(pot).cuda()
    tl = torch.from_numpy(lens).cuda()
    say(f"{name}: GPU marginals B={B} N={E + 1} C={C}")
    z, m = binding.marginals(tp, tl)
    torch.cuda.synchronize()
    say(f"{name}: oracle log Z")
    zo = oracle.logpartition(pot, lens)
    check_logz(z.cpu().numpy(), zo)
    # every valid edge sums to one; padding is exactly zero
    s = m.double().sum(dim=(2, 3)).cpu().numpy()
    for b in range(B):
        Eb = int(lens[b]) - 1
        assert np.abs(s[b, :Eb] - 1).max() < 1e-4
        assert torch.count_nonzero(m[b, Eb:]).item() == 0
    # sampled edges, checked element by element
    rng = np.random.default_rng(5)
    for b in sorted(set([0, B - 1, int(rng.integers(B))])):
        Eb = int(lens[b]) - 1
        for t0 in sorted(set([0, Eb // 2, max(0, Eb - 3)])):
            t1 = min(t0 + 3, E)
            say(f"{name}: oracle marginals b={b} edges [{t0},{t1})")
            ref, zb = oracle.marginals_seq(pot, lens, b, t0, t1)
            got = m[b, t0:t1].cpu().numpy().astype(np.float64)
            err = np.abs(got - ref).max()
            assert err <= MARG_ATOL, f"b={b} t=[{t0},{t1}) max abs err {err:.3e}"
    del m
    say(f"{name}: GPU Viterbi")
    path, score = binding.viterbi(tp, tl)
    torch.cuda.synchronize()
    say(f"{name}: oracle Viterbi")
    po, so = oracle.viterbi(pot, lens)
    check_logz(score.cpu().numpy(), so, "score")
    pg = path.cpu().numpy()
    bad = np.nonzero((pg != po).any(1))[0]
    assert bad.size == 0, f"Viterbi path mismatch in sequences {bad}"

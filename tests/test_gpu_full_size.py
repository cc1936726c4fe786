"""Parity at the full sizes of the larger workloads (B=32 N=512 C=64, B=16 N=1024 C=256,
B=4 N=8192 C=128, and B=33 N=1024 C=256, past 2^31 elements per array), in the launch
configuration the benchmark uses: log Z and Viterbi path and score of every sequence, and
the marginals of EVERY edge of every sequence, element by element, against the float64
oracle's forward-backward messages streamed edge range by edge range (the marginal tensor
is never held in float64 at once).
Padding edges must be exactly 0.  The combined marginals + Viterbi call must reproduce
the separate calls bitwise."""
import numpy as np
import pytest

from gpu_util import MARG_ATOL, check_logz, say
from paper_2002_00876_amd import workloads as W

pytestmark = pytest.mark.gpu

CHUNK_FLOATS = 1 << 22        # edges compared per oracle call: about 32 MB of float64


def compare_every_edge(m, pot, lens, name):
    """Max abs error of the GPU marginals m (a torch tensor [B, E, C, C] on the device)
    over every valid edge, against the oracle; padding checked to be exactly 0."""
    import torch

    import oracle

    B, E, C, _ = pot.shape
    say(f"{name}: oracle forward-backward messages")
    msg = oracle.Messages(pot, lens)
    chunk = max(1, CHUNK_FLOATS // (C * C))
    buf = np.empty((chunk, C, C), np.float64)
    worst, where = 0.0, None
    for b in range(B):
        Eb = int(lens[b]) - 1
        assert torch.count_nonzero(m[b, Eb:]).item() == 0, f"{name}: padding of sequence {b}"
        for t0 in range(0, Eb, chunk):
            t1 = min(Eb, t0 + chunk)
            ref = msg.edge_marginals(b, t0, t1, out=buf[:t1 - t0])
            got = m[b, t0:t1].cpu().numpy()
            err = np.abs(got.astype(np.float64) - ref)
            e = float(err.max())
            if e > worst:
                worst = e
                where = (b, t0 + int(np.unravel_index(err.argmax(), err.shape)[0]))
        say(f"{name}: sequence {b} ({Eb} edges) compared; max abs err so far {worst:.3e}")
    return worst, where, msg.logz


# past 2^31 elements per array: the HMM-style construction with 33 sequences (2.21e9
# elements, 8.8 GB of potentials and as much of marginals)
PAST_2_31 = W.Workload("hmm_b33", 33, 1024, 256, seed=9, kind="hmm")


@pytest.mark.parametrize("workload", ["mid", "long", "hmm", PAST_2_31],
                         ids=["mid", "long", "hmm", "hmm_b33"])
def test_full_size(workload):
    import torch

    import oracle
    from paper_2002_00876_amd import binding

    name = workload if isinstance(workload, str) else workload.name
    say(f"{name}: generating")
    pot, lens = W.generate(workload)
    B, E, C, _ = pot.shape
    tp = torch.from_numpy(pot).cuda()
    tl = torch.from_numpy(lens).cuda()
    say(f"{name}: GPU marginals B={B} N={E + 1} C={C}")
    z, m = binding.marginals(tp, tl)
    torch.cuda.synchronize()
    worst, where, zo = compare_every_edge(m, pot, lens, name)
    check_logz(z.cpu().numpy(), zo)
    assert worst <= MARG_ATOL, f"{name}: marginals max abs err {worst:.3e} at (b, t) = {where}"
    say(f"{name}: every edge within {MARG_ATOL:g} (max {worst:.3e})")
    say(f"{name}: GPU Viterbi")
    path, score = binding.viterbi(tp, tl)
    torch.cuda.synchronize()
    say(f"{name}: combined call against the separate calls")
    z3, m3, p3, s3 = binding.marginals_viterbi(tp, tl)
    torch.cuda.synchronize()
    assert torch.equal(z3, z) and torch.equal(p3, path) and torch.equal(s3, score)
    assert torch.equal(m3, m), f"{name}: combined-call marginals differ from the separate call"
    del m, m3
    say(f"{name}: oracle Viterbi")
    po, so = oracle.viterbi(pot, lens)
    check_logz(score.cpu().numpy(), so, "score")
    pg = path.cpu().numpy()
    bad = np.nonzero((pg != po).any(1))[0]
    assert bad.size == 0, f"Viterbi path mismatch in sequences {bad}"

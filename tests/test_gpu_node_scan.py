"""GPU parity of log Z where the tree stops below the root and the recursion over a level's
nodes finishes the sequence (log Z alone, 64 < C <= 128): the stopping level follows the
length (pairs at N = 20, level 5 at N = 512, level 7 at N = 2049), with ragged lengths
down to one and two tokens, odd label counts (scalar loads), -inf entries and a wide
dynamic range.  Compared with the float64 oracle and with the marginals call's log Z
(which runs the tree to the root)."""
import numpy as np
import pytest

import oracle
from gpu_util import check_logz, say
from paper_2002_00876_amd import workloads as W

pytestmark = pytest.mark.gpu


def _both(pot, lens):
    import torch
    from paper_2002_00876_amd import binding
    dev = torch.device("cuda:0")
    tp = torch.from_numpy(np.ascontiguousarray(pot)).to(dev)
    tl = torch.from_numpy(np.ascontiguousarray(lens)).to(dev)
    z = binding.logpartition(tp, tl)
    z2, _ = binding.marginals(tp, tl)
    torch.cuda.synchronize()
    return z.cpu().numpy(), z2.cpu().numpy()


CASES = [  # (B, N, C, lengths, sigma)
    (4, 20, 100, [20, 11, 2, 1], 1.5),
    (3, 20, 80, [20, 19, 3], 1.5),
    (3, 40, 67, [40, 33, 17], 1.5),     # odd C: scalar node loads
    (2, 512, 128, [512, 301], 1.5),
    (2, 2049, 96, [2049, 1500], 1.5),
    (3, 100, 128, [100, 64, 5], 40.0),  # wide range: float64 vectors and row weights
]


@pytest.mark.parametrize("B,N,C,lens,sigma", CASES)
def test_node_scan_log_z(B, N, C, lens, sigma):
    pot, lens = W.random_case(9000 + N + C, B, N, C, sigma=sigma, lengths=lens)
    say(f"node scan B={B} N={N} C={C} sigma={sigma}")
    z, z2 = _both(pot, lens)
    zo = oracle.logpartition(pot, lens)
    check_logz(z, zo)
    check_logz(z, z2.astype(np.float64), "log Z: recursion over nodes vs tree to the root")


def test_node_scan_neg_inf():
    pot, lens = W.random_case(9100, 3, 30, 72, lengths=[30, 17, 4], neg_inf_frac=0.3)
    pot[1, 5] = -np.inf            # sequence 1 has no finite path
    pot[2, 0, :, :36] = -np.inf    # half the labels cannot be entered at edge 0
    z, _ = _both(pot, lens)
    check_logz(z, oracle.logpartition(pot, lens))

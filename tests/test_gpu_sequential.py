"""GPU parity of the left-to-right forward kernel (ts_chain_logpartition_sequential) with
the float64 oracle, on both of its variants (one wave per sequence for C <= 64, one
workgroup per sequence above), and its agreement with the scan."""
import numpy as np
import pytest

import oracle
from gpu_util import check_logz, say
from paper_2002_00876_amd import workloads as W

pytestmark = pytest.mark.gpu


def _seq(pot, lens):
    import torch
    from paper_2002_00876_amd import binding
    dev = torch.device("cuda:0")
    tp = torch.from_numpy(np.ascontiguousarray(pot)).to(dev)
    tl = torch.from_numpy(np.ascontiguousarray(lens)).to(dev)
    z = binding.logpartition_sequential(tp, tl)
    zs = binding.logpartition(tp, tl)
    torch.cuda.synchronize()
    return z.cpu().numpy(), zs.cpu().numpy()


@pytest.mark.parametrize("C", [1, 3, 8, 20, 33, 64, 65, 130, 256])
def test_sequential_matches_oracle(C):
    N = 40 if C <= 130 else 12
    pot, lens = W.random_case(700 + C, 4, N, C, sigma=1.5)
    say(f"sequential C={C} N={N}")
    z, zs = _seq(pot, lens)
    zo = oracle.logpartition(pot, lens)
    check_logz(z, zo, "log Z (sequential)")
    check_logz(z, zs.astype(np.float64), "sequential vs scan")


@pytest.mark.parametrize("name", ["tiny", "paper"])
def test_sequential_on_named_workloads(name):
    pot, lens = W.generate(name)
    z, _ = _seq(pot, lens)
    check_logz(z, oracle.logpartition(pot, lens), "log Z (sequential)")


def test_sequential_neg_inf_and_single_token():
    pot, lens = W.random_case(710, 4, 9, 5, neg_inf_frac=0.4, lengths=[1, 2, 9, 5])
    z, _ = _seq(pot, lens)
    check_logz(z, oracle.logpartition(pot, lens), "log Z (sequential, -inf entries)")

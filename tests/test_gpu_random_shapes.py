"""Parity on seeded random shapes: label counts across every path of the library (the
single-launch kernels, the chunk path at C <= 64, the tree with 64- and 128-wide tiles, odd
C), chain lengths up to about 1200 tokens, batch sizes 1 to 6, ragged and very short
lengths, and three value distributions (Gaussian potentials of scale 0.3 to 10, integer
ties, 30% of entries -inf).  Every case runs the three calls and the combined call against
the float64 oracle (log Z and score 1e-5 relative, marginals 1e-5 absolute, Viterbi paths
exact).  Scale-40 potentials are left to the fixed cases elsewhere and to the limit
recorded below: over long chains the float32 intermediate log values reach about 1.1e-5
on some of them."""
import numpy as np
import pytest

from gpu_util import MARG_ATOL, check_all, gpu_all
from paper_2002_00876_amd import workloads as W

pytestmark = pytest.mark.gpu

LABELS = [1, 2, 3, 5, 8, 16, 20, 31, 32, 33, 48, 63, 64, 65, 96, 100, 127, 128, 129, 160,
          191, 192, 200, 255, 256]
N_CASES = 48


def make_case(i, seed0=92000):
    """Case i of the sweep: (pot, lengths, description), drawn from one seeded generator per
    case so that each case can be rerun on its own."""
    rng = np.random.default_rng(seed0 + i)
    C = int(rng.choice(LABELS))
    budget = 2e7
    kind = str(rng.choice(["normal", "normal", "normal", "int", "neginf"]))
    max_n = int(max(2, min(1200, budget / (C * C))))
    N = int(rng.integers(1, max_n + 1))
    B = int(rng.integers(1, 7))
    B = max(1, min(B, int(budget // (N * C * C))))
    mode = str(rng.choice(["random", "full", "short"]))
    if mode == "short":
        lens = rng.integers(1, min(N, 4) + 1, size=B)
        lens[0] = N
    else:
        lens = mode
    seed = seed0 + 1000 + i
    if kind == "normal":
        sigma = float(rng.choice([0.3, 1.0, 2.0, 5.0, 10.0]))
        pot, lens = W.random_case(seed, B, N, C, sigma=sigma, lengths=lens)
        what = f"normal sigma={sigma}"
    elif kind == "int":
        pot, lens = W.random_case(seed, B, N, C, kind="int", int_range=1, lengths=lens)
        what = "integer ties"
    else:
        pot, lens = W.random_case(seed, B, N, C, sigma=1.0, lengths=lens, neg_inf_frac=0.3)
        what = "30% -inf"
    return pot, lens, f"#{i} B={B} N={N} C={C} {what}"


@pytest.mark.parametrize("i", range(N_CASES))
def test_random_shape(i):
    pot, lens, tag = make_case(i)
    check_all(pot, lens, tag)


@pytest.mark.xfail(strict=False, reason=(
    "scale-40 potentials over more than 1000 edges: float32 storage of the tree's (or the "
    "chunks') intermediate log values limits the marginals to about 1.1e-5 absolute"))
def test_scale40_long_chain_limit():
    # a chain of 1032 edges (log Z about 1.2e5) whose best path is contested by two families
    # of paths with probabilities 0.31 and 0.69 over about 25 edges: those marginals follow
    # the difference of the two families' scores, which the float32 intermediate log values
    # carry to about 5e-5 (1.06e-5 in the marginals, far above the float64 oracle's error)
    pot, lens = W.random_case(90051, 1, 1033, 128, sigma=40.0, lengths="full")
    _, _, m, _, _ = gpu_all(pot, lens)
    import oracle
    _, mo = oracle.marginals(pot, lens)
    err = float(np.abs(m.astype(np.float64) - mo).max())
    assert err <= MARG_ATOL, f"marginals: max abs err {err:.3e}"

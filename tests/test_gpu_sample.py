"""GPU parity of forward-filtering backward-sampling against the float64 oracle, both fed
the same caller uniforms, on both paths (single launch and multi-launch tree).

The draws are integers decided by floating point: the GPU takes them from fp32 marginals
by an fp32 inverse CDF, the oracle from fp64 ones.  The two can differ only where u * total
falls within the GPU's error of a bin edge.  That error, relative to the total, is bounded
by the fp32 prefix sum of at most C <= 256 non-negative weights (C * 2^-24 <= 1.5e-5) plus
the weights' own relative error (the marginals' ~1e-6), so MARGIN_TOL = 2e-5: every
sequence whose GPU path differs from the oracle's must have an oracle draw margin (distance
of u * total from the nearest bin edge, relative to the total) below it, and such
sequences must be rare.  Every drawn transition must have a finite
potential, and closed forms (uniform potentials give floor(u * C)) hold exactly.
"""
import numpy as np
import pytest

import oracle
from gpu_util import say
from paper_2002_00876_amd import workloads as W

pytestmark = pytest.mark.gpu

MARGIN_TOL = 2e-5
MAX_DIFF_FRAC = 0.02


@pytest.fixture(params=["auto", "tree"], autouse=True)
def path_mode(request, monkeypatch):
    if request.param == "tree":
        monkeypatch.setenv("TS_PATH", "tree")
    else:
        monkeypatch.delenv("TS_PATH", raising=False)
    return request.param


def _gpu_sample(pot, lens, u):
    import torch
    from paper_2002_00876_amd import binding
    dev = torch.device("cuda:0")
    tp = torch.from_numpy(np.ascontiguousarray(pot)).to(dev)
    tl = torch.from_numpy(np.ascontiguousarray(lens)).to(dev)
    tu = torch.from_numpy(np.ascontiguousarray(u)).to(dev)
    z = binding.sample(tp, tu, tl)
    torch.cuda.synchronize()
    return z.cpu().numpy()


def _uniforms(seed, S, B, N):
    return np.random.default_rng(seed).random((S, B, N), dtype=np.float32)


def _check_valid(z, pot, lens):
    S, B, N = z.shape
    C = pot.shape[2]
    for b in range(B):
        L = int(lens[b])
        assert np.all(z[:, b, L:] == -1), "padding is not -1"
        zb = z[:, b, :L]
        assert zb.min() >= 0 and zb.max() < C, "label out of range"
        if L > 1:
            t = np.arange(L - 1)
            w = pot[b, t[None, :], zb[:, :-1], zb[:, 1:]]
            assert np.all(np.isfinite(w)), "a drawn transition has potential -inf"


def _check_parity(pot, lens, u, tag):
    say(f"sample case {tag}: pot {pot.shape}, S={u.shape[0]}")
    z = _gpu_sample(pot, lens, u)
    _check_valid(z, pot, lens)
    zo, margin = oracle.sample(pot, u, lens)
    diff = np.any(z != zo, axis=2)
    if diff.any():
        worst = margin[diff].max()
        assert worst < MARGIN_TOL, (
            f"{diff.sum()} sequences differ; one has oracle margin {worst:.2e}")
    assert diff.mean() <= MAX_DIFF_FRAC, f"{diff.mean():.3f} of the sequences differ"
    say(f"  {diff.sum()} of {diff.size} sampled sequences differ (all at bin edges; worst "
        f"oracle margin {margin[diff].max(initial=0.0):.2e})")
    return z


@pytest.mark.parametrize("seed", range(6))
def test_random_cases(seed):
    rng = np.random.default_rng(700 + seed)
    C = int(rng.choice([1, 3, 8, 20, 33, 64, 65, 130]))
    N = int(rng.integers(1, 40))
    B = 4
    pot, lens = W.random_case(seed + 800, B, N, C, sigma=float(rng.choice([0.5, 1.0, 3.0])))
    _check_parity(pot, lens, _uniforms(seed, 16, B, N), f"seed {seed} C={C} N={N}")


@pytest.mark.parametrize("name", ["tiny", "paper"])
def test_named_workloads(name):
    pot, lens = W.generate(name)
    B, E, C, _ = pot.shape
    _check_parity(pot, lens, _uniforms(11, 64, B, E + 1), name)


def test_largest_label_count_tree():
    # C = 256 spans all four register chunks of a draw
    pot, lens = W.random_case(901, 2, 12, 256, sigma=2.0)
    _check_parity(pot, lens, _uniforms(12, 8, 2, 12), "C=256")


def test_uniform_potentials_give_floor_u_c():
    B, N, C = 3, 9, 7
    pot = np.zeros((B, N - 1, C, C), np.float32)
    lens = np.array([9, 5, 1], np.int32)
    rng = np.random.default_rng(5)
    # centres of the bins, jittered by at most a quarter bin: no rounding can cross an edge
    k = rng.integers(0, C, size=(4, B, N))
    u = ((k + 0.5 + rng.uniform(-0.25, 0.25, size=k.shape)) / C).astype(np.float32)
    z = _gpu_sample(pot, lens, u)
    for b in range(B):
        L = int(lens[b])
        assert np.array_equal(z[:, b, :L], k[:, b, :L]), "uniform draws are not floor(u C)"
        assert np.all(z[:, b, L:] == -1)


def test_forbidden_transitions_are_never_drawn():
    rng = np.random.default_rng(9)
    B, N, C = 4, 30, 12
    pot, lens = W.random_case(902, B, N, C, sigma=1.0)
    mask = rng.random(pot.shape) < 0.6
    eye = np.eye(C, dtype=bool)[None, None]
    pot = np.where(mask & ~eye, -np.inf, pot).astype(np.float32)   # the diagonal stays open
    _check_parity(pot, lens, _uniforms(13, 32, B, N), "masked")


def test_single_token_sequences():
    B, N, C = 3, 1, 5
    pot = np.zeros((B, 0, C, C), np.float32)
    lens = np.ones(B, np.int32)
    u = np.array([[[0.0], [0.5], [0.99]]], np.float32)
    z = _gpu_sample(pot, lens, u)
    assert z.reshape(-1).tolist() == [0, 2, 4]

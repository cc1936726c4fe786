"""Pins of the oracle's forward-filtering backward-sampling against facts that do not come
from the oracle: the empirical distribution of many draws against p(z) by enumeration,
closed forms of the inverse-CDF convention (uniform potentials give z_t = floor(u_t C)),
a one-edge categorical worked by hand, and planted mistakes that must fail them."""
import math
import os

import numpy as np
import pytest

import oracle
from brute import enumerate_seq
from paper_2002_00876_amd import workloads as W

SRC = os.path.join(os.path.dirname(oracle.__file__), "oracle.c")


def _empirical_vs_exact(pot, L, paths, C):
    """(max |freq - p| / sigma over all sequences, number of distinct sequences drawn)."""
    seqs = enumerate_seq(pot[0], L, C)
    scores = np.array([s for _, s in seqs])
    p = np.exp(scores - scores.max())
    p /= p.sum()
    index = {z: k for k, (z, _) in enumerate(seqs)}
    counts = np.zeros(len(seqs))
    for z in paths[:, 0, :L]:
        counts[index[tuple(int(v) for v in z)]] += 1
    S = len(paths)
    sigma = np.sqrt(p * (1 - p) / S) + 1e-12
    return np.max(np.abs(counts / S - p) / sigma)


def test_draws_follow_the_chain_distribution():
    pot, lens = W.random_case(21, 1, 4, 3, lengths="full")
    S = 20000
    u = np.random.default_rng(5).random((S, 1, 4), dtype=np.float32)
    paths, _ = oracle.sample(pot, u, lens)
    assert _empirical_vs_exact(pot, 4, paths, 3) < 5.0


def test_uniform_potentials_give_floor_u_c():
    C, N = 5, 6
    pot = np.zeros((2, N - 1, C, C), np.float32)
    lens = np.array([N, 3], np.int32)
    u = np.random.default_rng(6).random((7, 2, N), dtype=np.float32)
    paths, _ = oracle.sample(pot, u, lens)
    want = np.floor(u.astype(np.float64) * C).astype(np.int32)
    want[:, 1, 3:] = -1
    np.testing.assert_array_equal(paths, want)


def test_single_token_is_uniform():
    pot = np.zeros((3, 0, 4, 4), np.float32)
    u = np.array([[[0.0], [0.3], [0.99]]], np.float32)
    paths, _ = oracle.sample(pot, u)
    np.testing.assert_array_equal(paths[0, :, 0], [0, 1, 3])


def test_one_edge_by_hand():
    pot, lens = W.random_case(22, 1, 2, 3, lengths="full")
    p = np.exp(pot[0, 0].astype(np.float64))
    p /= p.sum()                                        # joint of (z_0, z_1)
    u = np.array([[[0.61, 0.37]]], np.float32)          # u[0] draws z_0, u[1] draws z_1
    col = p.sum(axis=0)
    z1 = int(np.searchsorted(np.cumsum(col), 0.37 * col.sum(), side="right"))
    cond = p[:, z1]
    z0 = int(np.searchsorted(np.cumsum(cond), 0.61 * cond.sum(), side="right"))
    paths, margin = oracle.sample(pot, u, lens)
    np.testing.assert_array_equal(paths[0, 0], [z0, z1])
    assert margin[0, 0] > 0


def test_dominant_path_is_always_drawn():
    det = np.full((1, 5, 3, 3), -40.0, np.float32)
    for t in range(5):
        det[0, t, (t + 2) % 3, (t + 3) % 3] = 40.0
    u = np.random.default_rng(7).random((50, 1, 6), dtype=np.float32)
    paths, _ = oracle.sample(det, u)
    want = [(t + 2) % 3 for t in range(6)]
    assert all(list(p[0]) == want for p in paths)


MUTANTS = {
    "row_instead_of_column": ("for (int64_t i = 0; i < C; ++i) w[i] = mu[i * C + z[t + 1]];",
                              "for (int64_t i = 0; i < C; ++i) w[i] = mu[z[t + 1] * C + i];"),
    "last_token_from_row_sums": ("for (int64_t i = 0; i < C; ++i) w[j] += mu[i * C + j];",
                                 "for (int64_t i = 0; i < C; ++i) w[j] += mu[j * C + i];"),
    "uniform_index_shifted": ("z[t] = draw(w, C, (double)u[t], &d);",
                              "z[t] = draw(w, C, (double)u[t + 1], &d);"),
    "inclusive_bound": ("if (cum > x || k == C - 1) {", "if (cum >= x || k == C - 1) {"),
}


def _pins_pass(lib):
    pot, lens = W.random_case(21, 1, 4, 3, lengths="full")
    u = np.random.default_rng(5).random((20000, 1, 4), dtype=np.float32)
    paths, _ = oracle.sample(pot, u, lens, lib=lib)
    if not _empirical_vs_exact(pot, 4, paths, 3) < 5.0:
        return False
    C, N = 4, 6
    z0 = np.zeros((2, N - 1, C, C), np.float32)
    uu = np.random.default_rng(6).random((7, 2, N), dtype=np.float32)
    uu[0, 0, :] = [0.0, 0.25, 0.5, 0.75, 0.0, 0.25]  # exact bin edges: pins the strict rule
    paths, _ = oracle.sample(z0, uu, None, lib=lib)
    return np.array_equal(paths, np.floor(uu.astype(np.float64) * C).astype(np.int32))


def test_unmodified_sampler_passes(tmp_path):
    lib = oracle.load_library(oracle.compile_source(SRC, str(tmp_path / "liborc.so")))
    assert _pins_pass(lib)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_sampler_mistake_is_caught(tmp_path, name):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) >= 1, f"mutation site for {name} not found"
    path = tmp_path / "oracle_mutant.c"
    path.write_text(src.replace(old, new, 1))
    lib = oracle.load_library(oracle.compile_source(str(path), str(tmp_path / "libmut.so")))
    assert not _pins_pass(lib), f"pins did not catch mutant {name}"

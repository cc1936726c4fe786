"""Pins of the oracle's entropy and log-density (the chain distribution's entropy, Table 2
"Entropy" semiring; log p(z) of one structure, Sec. 5.1) against facts that do not come
from the oracle: enumeration of every label sequence, closed forms and invariants.  A
planted mistake in the entropy's chain-rule terms must fail them."""
import math
import os

import numpy as np
import pytest
from scipy.stats import entropy as scipy_entropy

import oracle
from brute import brute_entropy, brute_log_density, enumerate_seq
from paper_2002_00876_amd import workloads as W

SRC = os.path.join(os.path.dirname(oracle.__file__), "oracle.c")


def _cases():
    for seed in range(8):
        rng = np.random.default_rng(300 + seed)
        C = int(rng.integers(1, 5))
        N = int(rng.integers(1, 7))
        kind = "int" if seed % 2 else "normal"
        yield W.random_case(seed + 40, 3, N, C, kind=kind, lengths=[1, min(2, N), N])


@pytest.mark.parametrize("case", range(8))
def test_entropy_matches_enumeration(case):
    pot, lens = list(_cases())[case]
    np.testing.assert_allclose(oracle.entropy(pot, lens), brute_entropy(pot, lens),
                               rtol=1e-11, atol=1e-12)


def test_entropy_of_tiny_workload():
    pot, lens = W.generate("tiny")
    np.testing.assert_allclose(oracle.entropy(pot, lens), brute_entropy(pot, lens), rtol=1e-12)


@pytest.mark.parametrize("C,N", [(1, 4), (3, 1), (3, 5), (7, 9)])
def test_entropy_of_zero_potentials_is_uniform(C, N):
    # every one of the C**L sequences is equally likely: H = L log C
    pot = np.zeros((2, max(N - 1, 0), C, C), np.float32)
    lens = np.array([N, max(1, N - 2)], np.int32)
    np.testing.assert_allclose(oracle.entropy(pot, lens), lens * math.log(C), rtol=1e-13,
                               atol=1e-13)


def test_one_edge_entropy_is_a_categorical_entropy():
    pot, lens = W.random_case(7, 4, 2, 5, lengths="full")
    want = [scipy_entropy(np.exp(pot[b, 0].astype(np.float64).ravel()
                                 - pot[b, 0].astype(np.float64).max())) for b in range(4)]
    np.testing.assert_allclose(oracle.entropy(pot, lens), want, rtol=1e-12)


def test_entropy_bounds_and_near_deterministic_chain():
    pot, lens = W.random_case(9, 6, 8, 4, sigma=2.0)
    H = oracle.entropy(pot, lens)
    assert np.all(H >= 0) and np.all(H <= lens * math.log(4) + 1e-12)
    # one path 60 nats above every other: H is essentially 0
    det = np.full((1, 5, 3, 3), -30.0, np.float32)
    for t in range(5):
        det[0, t, t % 3, (t + 1) % 3] = 30.0
    assert oracle.entropy(det, np.array([6], np.int32))[0] < 1e-20


@pytest.mark.parametrize("case", range(8))
def test_log_density_matches_enumeration(case):
    pot, lens = list(_cases())[case]
    B, E, C, _ = pot.shape
    rng = np.random.default_rng(case)
    labels = rng.integers(0, C, size=(B, E + 1)).astype(np.int32)
    got = oracle.log_density(pot, labels, lens)
    want = brute_log_density(pot, lens, labels)
    fin = np.isfinite(want)
    np.testing.assert_allclose(got[fin], want[fin], rtol=1e-11, atol=1e-12)
    assert np.array_equal(np.isneginf(got), np.isneginf(want))


def test_densities_of_all_sequences_sum_to_one():
    pot, lens = W.random_case(11, 1, 5, 3, lengths="full")
    seqs = enumerate_seq(pot[0], 5, 3)
    labels = np.array([z for z, _ in seqs], np.int32)
    lp = np.array([oracle.log_density(pot, z[None], lens)[0] for z in labels])
    assert abs(np.exp(lp).sum() - 1.0) < 1e-12


def test_log_density_of_zero_potentials():
    pot = np.zeros((2, 4, 3, 3), np.float32)
    lens = np.array([5, 2], np.int32)
    labels = np.array([[0, 1, 2, 0, 1], [2, 2, -7, 99, 5]], np.int32)   # past length: ignored
    np.testing.assert_allclose(oracle.log_density(pot, labels, lens), -lens * math.log(3),
                               rtol=1e-14)


def test_log_density_rejects_out_of_range_labels():
    pot = np.zeros((1, 2, 3, 3), np.float32)
    with pytest.raises(ValueError):
        oracle.log_density(pot, np.array([[0, 3, 1]], np.int32))


MUTANTS = {
    "entropy_drops_first_node_term": ("if (t == 0) h -= m * log(m);", "(void)0;"),
    "entropy_joint_not_conditional": (
        "h -= mu[i * C + j] * log(mu[i * C + j] / m);", "h -= mu[i * C + j] * log(mu[i * C + j]);"),
    "entropy_node_term_every_edge": ("if (t == 0) h -= m * log(m);", "h -= m * log(m);"),
    "density_drops_log_z": ("out[b] = s - logZ[b];", "out[b] = s;"),
    "density_transposed_gather": ("pot_at(pf, pd, N, C, b, t, z[t], z[t + 1]);",
                                  "pot_at(pf, pd, N, C, b, t, z[t + 1], z[t]);"),
}


def _pins_pass(lib):
    for pot, lens in [W.random_case(s, 3, 5, 3, kind=k, lengths=[5, 3, 2]) for s, k in
                      [(1, "normal"), (2, "int")]]:
        if not np.allclose(oracle.entropy(pot, lens, lib=lib), brute_entropy(pot, lens),
                           rtol=1e-11):
            return False
        labels = np.random.default_rng(0).integers(0, 3, size=(3, 5)).astype(np.int32)
        if not np.allclose(oracle.log_density(pot, labels, lens, lib=lib),
                           brute_log_density(pot, lens, labels), rtol=1e-11):
            return False
    return True


def test_unmodified_entropy_oracle_passes(tmp_path):
    lib = oracle.load_library(oracle.compile_source(SRC, str(tmp_path / "liborc.so")))
    assert _pins_pass(lib)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_entropy_mistake_is_caught(tmp_path, name):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) >= 1, f"mutation site for {name} not found"
    path = tmp_path / "oracle_mutant.c"
    path.write_text(src.replace(old, new, 1))
    lib = oracle.load_library(oracle.compile_source(str(path), str(tmp_path / "libmut.so")))
    assert not _pins_pass(lib), f"pins did not catch mutant {name}"

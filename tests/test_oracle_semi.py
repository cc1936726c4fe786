"""Pins of the oracle's semi-Markov CRF (Table 1, "Semi-Markov": segment labels, parts
N K C^2, segmental forward-backward) against facts that do not come from the oracle:

- brute-force enumeration of every labelled segmentation on tiny cases, including integer
  potentials with exact ties, -inf entries and one-token sequences;
- K = 1 is the linear chain, whose oracle is pinned separately;
- closed forms of zero potentials: with K >= E every composition of E is allowed, so
  Z = C^2 (1 + C)^(E-1); with C = 1 and K = 2, Z is the Fibonacci number F(E+1);
- invariants: every step is covered by exactly one segment, a segment starts at step 0,
  and a segment ends with label j exactly where one starts after j;
- central finite differences of log Z against the marginals (float64 entry point);
- planted mistakes in a copy of the source must fail these pins.
"""
import math
import os

import numpy as np
import pytest

import oracle
from brute import brute_semi

SRC = os.path.join(os.path.dirname(oracle.__file__), "oracle.c")


def semi_case(seed, B, N, K, C, kind="normal", lengths=None, neg_inf_frac=0.0, sigma=1.0):
    rng = np.random.default_rng(seed)
    shape = (B, N - 1, K, C, C)
    if kind == "normal":
        sp = rng.standard_normal(shape) * sigma
    else:
        sp = rng.integers(-1, 1, endpoint=True, size=shape).astype(np.float64)
    if neg_inf_frac:
        sp[rng.random(shape) < neg_inf_frac] = -np.inf
    lens = (rng.integers(1, N, endpoint=True, size=B) if lengths is None
            else np.asarray(lengths))
    return sp.astype(np.float32), lens.astype(np.int32)


BRUTE_CASES = [
    (1, 3, 6, 3, 2, "normal", [6, 4, 1]),
    (2, 3, 5, 2, 3, "normal", [5, 2, 3]),
    (3, 2, 6, 5, 2, "normal", [6, 5]),
    (4, 3, 5, 3, 2, "int", [5, 5, 4]),
    (5, 2, 6, 2, 2, "int", [6, 3]),
    (6, 2, 5, 1, 3, "normal", [5, 4]),
]


@pytest.mark.parametrize("case", BRUTE_CASES, ids=lambda c: f"seed{c[0]}")
def test_semi_matches_enumeration(case):
    seed, B, N, K, C, kind, lens = case
    sp, lens = semi_case(seed, B, N, K, C, kind, lens)
    zb, mb, sb, pb, gb = brute_semi(sp, lens)
    zo, mo = oracle.semi_marginals(sp, lens)
    po, go, so = oracle.semi_viterbi(sp, lens)
    np.testing.assert_allclose(zo, zb, rtol=1e-12)
    np.testing.assert_allclose(mo, mb, atol=1e-12)
    np.testing.assert_allclose(so, sb, rtol=1e-12)
    np.testing.assert_array_equal(po, pb)
    np.testing.assert_array_equal(go, gb)


def test_semi_with_forbidden_entries_matches_enumeration():
    sp, lens = semi_case(7, 4, 5, 3, 2, "normal", [5, 4, 3, 2], neg_inf_frac=0.5)
    zb, mb, sb, pb, gb = brute_semi(sp, lens)
    zo, mo = oracle.semi_marginals(sp, lens)
    po, go, so = oracle.semi_viterbi(sp, lens)
    np.testing.assert_array_equal(np.isneginf(zo), np.isneginf(zb))
    fin = np.isfinite(zb)
    np.testing.assert_allclose(zo[fin], zb[fin], rtol=1e-12)
    np.testing.assert_allclose(mo, mb, atol=1e-12)
    np.testing.assert_array_equal(so, sb)
    np.testing.assert_array_equal(po[fin], pb[fin])
    np.testing.assert_array_equal(go[fin], gb[fin])


def test_k1_is_the_linear_chain():
    sp, lens = semi_case(8, 5, 9, 1, 4, "normal", [9, 7, 2, 1, 5])
    zs, ms = oracle.semi_marginals(sp, lens)
    ps, gs, ss = oracle.semi_viterbi(sp, lens)
    pot = sp[:, :, 0]
    zc, mc = oracle.marginals(pot, lens)
    pc, sc = oracle.viterbi(pot, lens)
    np.testing.assert_allclose(zs, zc, rtol=1e-13)
    np.testing.assert_allclose(ms[:, :, 0], mc, atol=1e-13)
    np.testing.assert_array_equal(ps, pc)
    np.testing.assert_array_equal(ss, sc)
    for b, L in enumerate(lens):
        assert np.all(gs[b, :L - 1] == 1) and np.all(gs[b, L - 1:] == -1)


@pytest.mark.parametrize("E,C", [(1, 3), (4, 2), (6, 5)])
def test_zero_potentials_all_compositions(E, C):
    sp = np.zeros((1, E, E, C, C), np.float32)            # K = E: every composition
    want = 2 * math.log(C) + (E - 1) * math.log(1 + C)
    np.testing.assert_allclose(oracle.semi_logpartition(sp), [want], rtol=1e-13)


@pytest.mark.parametrize("E", [1, 2, 5, 12])
def test_zero_potentials_fibonacci(E):
    sp = np.zeros((1, E, 2, 1, 1), np.float32)            # C = 1, K = 2
    fib = [1, 1]
    while len(fib) <= E + 1:
        fib.append(fib[-1] + fib[-2])
    np.testing.assert_allclose(oracle.semi_logpartition(sp), [math.log(fib[E])], rtol=1e-13)


def test_single_token_is_log_c():
    sp = np.zeros((2, 3, 2, 5, 5), np.float32)
    z = oracle.semi_logpartition(sp, np.array([1, 1], np.int32))
    np.testing.assert_allclose(z, [math.log(5)] * 2, rtol=1e-15)
    path, seglen, score = oracle.semi_viterbi(sp, np.array([1, 1], np.int32))
    assert path[:, 0].tolist() == [0, 0] and np.all(path[:, 1:] == -1)
    assert np.all(seglen == -1) and score.tolist() == [0.0, 0.0]


def test_coverage_and_flow_invariants():
    sp, lens = semi_case(9, 4, 14, 4, 3, "normal", [14, 9, 5, 2], sigma=2.0)
    _, mu = oracle.semi_marginals(sp, lens)
    B, E1, K, C, _ = mu.shape
    for b in range(B):
        E = int(lens[b]) - 1
        m = mu[b]
        assert np.all(m >= -1e-15) and np.all(m[E:] == 0)
        assert abs(m[0].sum() - 1) < 1e-12                    # a segment starts at step 0
        for s in range(E):                                    # each step covered once
            cov = sum(m[t, k - 1].sum() for t in range(E) for k in range(1, K + 1)
                      if t <= s < t + k)
            assert abs(cov - 1) < 1e-12
        for e in range(1, E):                                 # flow at each boundary
            ends = sum(m[e - k, k - 1].sum(axis=0) for k in range(1, min(K, e) + 1))
            starts = m[e].sum(axis=(0, 2))
            np.testing.assert_allclose(ends, starts, atol=1e-12)
        for t in range(E):                                    # nothing overruns the end
            for k in range(1, K + 1):
                if t + k > E:
                    assert np.all(m[t, k - 1] == 0)


def test_finite_differences_of_log_z():
    rng = np.random.default_rng(10)
    sp = rng.standard_normal((1, 5, 3, 2, 2))
    lens = np.array([6], np.int32)
    _, mu = oracle.semi_marginals(sp, lens)
    h = 1e-6
    for idx in [(0, 0, 0, 0, 1), (0, 2, 2, 1, 0), (0, 4, 0, 1, 1), (0, 1, 1, 0, 0)]:
        d = np.zeros_like(sp)
        d[idx] = h
        fd = (oracle.semi_logpartition(sp + d, lens) - oracle.semi_logpartition(sp - d, lens))
        np.testing.assert_allclose(fd[0] / (2 * h), mu[idx], atol=1e-8)


def test_viterbi_score_is_its_segmentation_score():
    sp, lens = semi_case(11, 6, 20, 4, 5, "normal", None, sigma=1.5)
    path, seglen, score = oracle.semi_viterbi(sp, lens)
    z = oracle.semi_logpartition(sp, lens)
    for b in range(len(lens)):
        E = int(lens[b]) - 1
        s, t = 0.0, 0
        while t < E:
            k = int(seglen[b, t])
            assert 1 <= k <= 4 and np.all(seglen[b, t + 1:t + k] == 0)
            assert np.all(path[b, t + 1:t + k + 1] == path[b, t + 1])
            s += float(sp[b, t, k - 1, path[b, t], path[b, t + 1]])
            t += k
        assert t == E
        assert s == pytest.approx(score[b], rel=1e-12)
        assert score[b] <= z[b] + 1e-12


MUTANTS = {
    "forward_length_index_wrapped": (
        "tmp[n++] = alpha[(e - k) * C + i] + sp_at(pf, pd, N, K, C, b, e - k, k - 1, i, j);",
        "tmp[n++] = alpha[(e - k) * C + i] + sp_at(pf, pd, N, K, C, b, e - k, k % K, i, j);"),
    "forward_transposed": (
        "tmp[n++] = alpha[(e - k) * C + i] + sp_at(pf, pd, N, K, C, b, e - k, k - 1, i, j);",
        "tmp[n++] = alpha[(e - k) * C + i] + sp_at(pf, pd, N, K, C, b, e - k, k - 1, j, i);"),
    "backward_drops_longest_segment": ("for (int64_t k = 1; k <= K && e + k <= E; ++k)",
                                       "for (int64_t k = 1; k < K && e + k <= E; ++k)"),
    "marginal_beta_at_start": ("+ beta[(e + k) * C + j] - A);", "+ beta[(e + 1) * C + j] - A);"),
    "longest_segment_on_ties": ("for (int64_t k = 1; k <= K && k <= e && !found; ++k)",
                                "for (int64_t k = (K < e ? K : e); k >= 1 && !found; --k)"),
    "seglen_at_segment_end": ("g[e - kb] = (int32_t)kb;", "g[e - 1] = (int32_t)kb;"),
    "max_segment_length_k_minus_one": ("for (int64_t k = 1; k <= K && k <= e; ++k)\n                for (int64_t i = 0; i < C; ++i)\n                    tmp",
                                       "for (int64_t k = 1; k < K && k <= e; ++k)\n                for (int64_t i = 0; i < C; ++i)\n                    tmp"),
}


def _pins_pass(lib):
    for case in BRUTE_CASES[:5]:
        seed, B, N, K, C, kind, lens = case
        sp, lens = semi_case(seed, B, N, K, C, kind, lens)
        zb, mb, sb, pb, gb = brute_semi(sp, lens)
        zo, mo = oracle.semi_marginals(sp, lens, lib=lib)
        po, go, so = oracle.semi_viterbi(sp, lens, lib=lib)
        if not (np.allclose(zo, zb, rtol=1e-12) and np.allclose(mo, mb, atol=1e-12)
                and np.allclose(so, sb, rtol=1e-12) and np.array_equal(po, pb)
                and np.array_equal(go, gb)):
            return False
    return True


def test_unmodified_semi_oracle_passes(tmp_path):
    lib = oracle.load_library(oracle.compile_source(SRC, str(tmp_path / "liborc.so")))
    assert _pins_pass(lib)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_semi_mistake_is_caught(tmp_path, name):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) >= 1, f"mutation site for {name} not found"
    path = tmp_path / "oracle_mutant.c"
    path.write_text(src.replace(old, new, 1))
    lib = oracle.load_library(oracle.compile_source(str(path), str(tmp_path / "libmut.so")))
    assert not _pins_pass(lib), f"pins did not catch mutant {name}"

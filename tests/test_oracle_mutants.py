"""The pins must be able to fail: each test plants one plausible mistake in a copy of
the oracle's C source (a transposed operand, a dropped term, a wrong index, a wrong tie
rule, a sign error), builds it on the CPU and checks that the pins reject it."""
import os

import numpy as np
import pytest

import oracle
from brute import brute
from paper_2002_00876_amd import workloads as W

SRC = os.path.join(os.path.dirname(oracle.__file__), "oracle.c")

MUTANTS = {
    "transposed_forward_operand": (
        "tmp[i] = alpha[t * C + i] + pot_at(pf, pd, N, C, b, t, i, j);",
        "tmp[i] = alpha[t * C + i] + pot_at(pf, pd, N, C, b, t, j, i);"),
    "dropped_last_edge": (
        "for (int64_t t = 0; t + 1 < L; ++t)\n        for (int64_t j = 0; j < C; ++j) {\n"
        "            for (int64_t i = 0; i < C; ++i)\n                tmp[i]",
        "for (int64_t t = 0; t + 2 < L; ++t)\n        for (int64_t j = 0; j < C; ++j) {\n"
        "            for (int64_t i = 0; i < C; ++i)\n                tmp[i]"),
    "beta_off_by_one_in_marginal": (
        "beta[(t + 1) * C + j] - logZ);", "beta[t * C + j] - logZ);"),
    "alpha_off_by_one_in_marginal": (
        "v = exp(alpha[t * C + i] +", "v = exp(alpha[(t + 1) * C + i] +"),
    "marginal_sign": ("beta[(t + 1) * C + j] - logZ);", "beta[(t + 1) * C + j] + logZ);"),
    "highest_index_ties": ("if (v > best) { best = v; arg = (int32_t)i; }",
                           "if (v >= best) { best = v; arg = (int32_t)i; }"),
    "backward_transposed": (
        "tmp[j] = pot_at(pf, pd, N, C, b, t, i, j) + beta[(t + 1) * C + j];",
        "tmp[j] = pot_at(pf, pd, N, C, b, t, j, i) + beta[(t + 1) * C + j];"),
    "lse_drops_shift": ("return m + log(s);", "return log(s);"),
}


def _pins_pass(lib):
    """A compact subset of the pins: brute force on random and tied cases."""
    cases = [W.random_case(s, 3, 5, 3, kind=k, lengths=[5, 3, 2], int_range=1)
             for s, k in [(1, "normal"), (2, "int"), (3, "normal"), (4, "int")]]
    for pot, lens in cases:
        zb, mb, sb, pb = brute(pot, lens)
        zo, mo = oracle.marginals(pot, lens, lib=lib)
        po, so = oracle.viterbi(pot, lens, lib=lib)
        if not (np.allclose(zo, zb, rtol=1e-12) and np.allclose(mo, mb, atol=1e-12)
                and np.allclose(so, sb, rtol=1e-12) and np.array_equal(po, pb)):
            return False
    return True


def test_unmodified_oracle_passes(tmp_path):
    lib = oracle.load_library(oracle.compile_source(SRC, str(tmp_path / "liborc.so")))
    assert _pins_pass(lib)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(tmp_path, name):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) >= 1, f"mutation site for {name} not found"
    mutated = src.replace(old, new, 1)
    path = tmp_path / "oracle_mutant.c"
    path.write_text(mutated)
    lib = oracle.load_library(oracle.compile_source(str(path), str(tmp_path / "libmut.so")))
    assert not _pins_pass(lib), f"pins did not catch mutant {name}"

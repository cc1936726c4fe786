"""Pins of the float64 oracle against facts that do not come from the oracle itself:
brute-force enumeration (Torch-Struct Sec. 5.1 footnote: enumerate all structures on small
sets), hand-derived fixtures, closed forms, invariants of the distribution, finite
differences of log Z (Sec. 5.1: marginals are dA/dl), and the tree-order evaluation of
Sec. 6a (associativity of the semiring product)."""
import math
import os

import numpy as np
import pytest
from scipy.special import logsumexp, softmax

import oracle
from brute import brute
from paper_2002_00876_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ----------------------------------------------------------------- brute force
@pytest.mark.parametrize("seed", range(12))
@pytest.mark.parametrize("kind", ["normal", "int"])
def test_oracle_matches_brute_force(seed, kind):
    rng = np.random.default_rng(100 + seed)
    C = int(rng.integers(1, 5))
    N = int(rng.integers(1, 8 if C <= 3 else 7))
    B = 3
    lens = np.array([1, min(2, N), N])[:B]
    pot, lens = W.random_case(seed, B, N, C, kind=kind, lengths=lens)
    zb, mb, sb, pb = brute(pot, lens)
    zo, mo = oracle.marginals(pot, lens)
    po, so = oracle.viterbi(pot, lens)
    np.testing.assert_allclose(zo, zb, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(mo, mb, rtol=0, atol=1e-12)
    np.testing.assert_allclose(so, sb, rtol=1e-12, atol=1e-12)
    np.testing.assert_array_equal(po, pb)


def test_tiny_workload_by_enumeration():
    pot, lens = W.generate("tiny")          # 2 sequences x 3^6 label sequences
    zb, mb, sb, pb = brute(pot, lens)
    zo, mo = oracle.marginals(pot, lens)
    po, so = oracle.viterbi(pot, lens)
    np.testing.assert_allclose(zo, zb, rtol=1e-13)
    np.testing.assert_allclose(mo, mb, atol=1e-13)
    np.testing.assert_allclose(so, sb, rtol=1e-13)
    np.testing.assert_array_equal(po, pb)


@pytest.mark.parametrize("seed", range(6))
def test_integer_ties_follow_lowest_index_backtrace(seed):
    # small integer potentials make many exactly tied maxima
    pot, lens = W.random_case(200 + seed, 4, 6, 3, kind="int", int_range=1, lengths="random")
    _, _, sb, pb = brute(pot, lens)
    po, so = oracle.viterbi(pot, lens)
    np.testing.assert_array_equal(so, sb)
    np.testing.assert_array_equal(po, pb)


def test_neg_inf_entries_against_brute_force():
    pot, lens = W.random_case(7, 4, 5, 3, kind="normal", lengths=[5, 4, 2, 1], neg_inf_frac=0.4)
    pot[0, 1] = -np.inf                      # sequence 0 has no finite path: log Z = -inf
    zb, mb, sb, pb = brute(pot, lens)
    zo, mo = oracle.marginals(pot, lens)
    po, so = oracle.viterbi(pot, lens)
    assert zo[0] == -np.inf and np.all(mo[0] == 0)
    np.testing.assert_allclose(zo, zb, rtol=1e-12)
    np.testing.assert_allclose(mo, mb, atol=1e-12)
    np.testing.assert_array_equal(so, sb)
    # with no finite sequence every path ties and only the backtrace fixes one (see the
    # no_finite_path fixture); elsewhere the reversed-lexicographic minimum is that path
    finite = np.isfinite(sb)
    np.testing.assert_array_equal(po[finite], pb[finite])


# ----------------------------------------------------------------- golden fixtures
def _parse_fixture(path):
    ns = {"e": math.e, "log": math.log, "exp": math.exp, "inf": math.inf}
    kv = {}
    for line in open(path):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        k, v = line.split(":", 1)
        kv[k.strip()] = v.strip()
    if "Z" in kv:
        ns["Z"] = eval(kv["Z"], {"__builtins__": {}}, ns)

    def tensor(s):
        return [[[eval(x, {"__builtins__": {}}, ns) for x in row.split()]
                 for row in edge.split("|")] for edge in s.split("||")]

    C, N = int(kv["C"]), int(kv["N"])
    pot = np.array(tensor(kv["pot"]), np.float64).reshape(1, N - 1, C, C)
    lens = np.array([int(kv["lengths"])], np.int32)
    out = dict(pot=pot, lens=lens,
               logZ=eval(kv["logZ"], {"__builtins__": {}}, ns),
               marg=np.array(tensor(kv["marg"]), np.float64).reshape(1, N - 1, C, C),
               score=eval(kv["score"], {"__builtins__": {}}, ns),
               path=np.array([int(x) for x in kv["path"].split()], np.int32))
    return out


@pytest.mark.parametrize("name", ["tie_2x2", "chain3", "padding", "single_token", "no_finite_path"])
def test_golden_fixture(name):
    fx = _parse_fixture(os.path.join(GOLDEN, name + ".txt"))
    zo, mo = oracle.marginals(fx["pot"], fx["lens"])          # float64 entry point
    po, so = oracle.viterbi(fx["pot"], fx["lens"])
    if math.isinf(fx["logZ"]):
        assert zo[0] == fx["logZ"] and so[0] == fx["score"]
    else:
        assert abs(zo[0] - fx["logZ"]) <= 1e-14 * max(1.0, abs(fx["logZ"]))
        assert abs(so[0] - fx["score"]) <= 1e-15
    np.testing.assert_allclose(mo, fx["marg"], atol=1e-15)
    np.testing.assert_array_equal(po[0], fx["path"])


# ----------------------------------------------------------------- closed forms
@pytest.mark.parametrize("C,N,L", [(1, 4, 4), (3, 7, 5), (8, 9, 9), (20, 25, 13)])
def test_zero_potentials(C, N, L):
    pot = np.zeros((2, N - 1, C, C), np.float32)
    lens = np.array([L, 1], np.int32)
    z, m = oracle.marginals(pot, lens)
    np.testing.assert_allclose(z, [L * math.log(C), math.log(C)], rtol=1e-14, atol=1e-14)
    np.testing.assert_allclose(m[0, :L - 1], 1.0 / C**2, rtol=1e-13)
    assert np.all(m[0, L - 1:] == 0) and np.all(m[1] == 0)
    p, s = oracle.viterbi(pot, lens)
    assert np.all(p[0, :L] == 0) and np.all(p[0, L:] == -1) and np.all(s == 0)


def test_first_label_independent_potentials():
    # l[t,i,j] = u_t[j]: the first label is free, each later label sums exp u_t independently
    rng = np.random.default_rng(3)
    B, N, C = 3, 9, 5
    u = rng.standard_normal((B, N - 1, C))
    pot = np.repeat(u[:, :, None, :], C, axis=2)
    lens = np.array([9, 4, 2], np.int32)
    z = oracle.logpartition(pot, lens)
    ref = [math.log(C) + sum(logsumexp(u[b, t]) for t in range(lens[b] - 1)) for b in range(B)]
    np.testing.assert_allclose(z, ref, rtol=1e-14)


def test_row_stochastic_potentials():
    # l[t,i,.] = log of a probability row: Z = sum over the first label of 1 = C
    rng = np.random.default_rng(4)
    B, N, C = 2, 12, 6
    T = rng.standard_normal((B, N - 1, C, C))
    pot = T - logsumexp(T, axis=3, keepdims=True)
    z = oracle.logpartition(pot, np.array([12, 7], np.int32))
    np.testing.assert_allclose(z, math.log(C), rtol=1e-14)


def test_single_label_chain():
    rng = np.random.default_rng(5)
    pot = rng.standard_normal((3, 10, 1, 1))
    lens = np.array([11, 6, 1], np.int32)
    z, m = oracle.marginals(pot, lens)
    p, s = oracle.viterbi(pot, lens)
    for b in range(3):
        ref = pot[b, :lens[b] - 1, 0, 0].sum()
        assert abs(z[b] - ref) < 1e-13 and abs(s[b] - ref) < 1e-13
        np.testing.assert_allclose(m[b, :lens[b] - 1], 1.0, atol=1e-14)
        assert np.all(m[b, lens[b] - 1:] == 0)
        assert np.all(p[b, :lens[b]] == 0)


def test_one_edge_is_a_categorical():
    # Sec. 5.1: A = LSE(l), dA/dl = softmax(l), A* = max(l), argmax indicator
    rng = np.random.default_rng(6)
    C = 7
    pot = rng.standard_normal((4, 1, C, C))
    z, m = oracle.marginals(pot, np.full(4, 2, np.int32))
    p, s = oracle.viterbi(pot, np.full(4, 2, np.int32))
    for b in range(4):
        assert abs(z[b] - logsumexp(pot[b, 0])) < 1e-13
        np.testing.assert_allclose(m[b, 0], softmax(pot[b, 0].ravel()).reshape(C, C), atol=1e-15)
        assert s[b] == pot[b, 0].max()
        i, j = np.unravel_index(np.argmax(pot[b, 0]), (C, C))
        assert (p[b, 0], p[b, 1]) == (i, j)


# ----------------------------------------------------------------- invariants
@pytest.mark.parametrize("seed", range(4))
def test_distribution_invariants(seed):
    pot, lens = W.random_case(300 + seed, 5, 40, 6, sigma=1.5, lengths="random")
    z, m = oracle.marginals(pot, lens)
    p, s = oracle.viterbi(pot, lens)
    for b in range(5):
        L = lens[b]
        if L > 1:
            np.testing.assert_allclose(m[b, :L - 1].sum(axis=(1, 2)), 1.0, atol=1e-12)
            # node consistency: incoming mass at a token = outgoing mass
            np.testing.assert_allclose(m[b, :L - 2].sum(axis=1), m[b, 1:L - 1].sum(axis=2), atol=1e-12)
        assert np.all(m[b] >= 0) and np.all(m[b] <= 1 + 1e-12)
        assert np.all(m[b, L - 1:] == 0)
        # A* <= A <= A* + L log C
        assert s[b] <= z[b] + 1e-12 and z[b] <= s[b] + L * math.log(6) + 1e-12
        own = sum(float(pot[b, t, p[b, t], p[b, t + 1]]) for t in range(L - 1))
        assert abs(own - s[b]) < 1e-12
        assert np.all(p[b, L:] == -1)


# ----------------------------------------------------------------- finite differences
def test_marginals_are_the_gradient_of_log_z():
    rng = np.random.default_rng(8)
    B, N, C = 2, 7, 4
    pot = rng.standard_normal((B, N - 1, C, C))
    lens = np.array([7, 5], np.int32)
    _, m = oracle.marginals(pot, lens)
    h = 1e-5
    for _ in range(40):
        b, t, i, j = (int(rng.integers(B)), int(rng.integers(N - 1)), int(rng.integers(C)),
                      int(rng.integers(C)))
        pp, pm = pot.copy(), pot.copy()
        pp[b, t, i, j] += h
        pm[b, t, i, j] -= h
        fd = (oracle.logpartition(pp, lens)[b] - oracle.logpartition(pm, lens)[b]) / (2 * h)
        assert abs(fd - m[b, t, i, j]) < 1e-8, (b, t, i, j, fd, m[b, t, i, j])


# ----------------------------------------------------------------- tree order (Sec. 6a)
def _tree_logz(pot_b, L, C, semiring):
    """log Z or max score by the balanced tree of Sec. 6a / Fig. 3: pad the edge list to a
    power of two with the identity I (0 on the diagonal, -inf elsewhere) and reduce pairs
    with the semiring matrix product (written with numpy, independent of the oracle)."""
    E = L - 1
    if E == 0:
        return math.log(C) if semiring == "log" else 0.0
    P = 1
    while P < E:
        P *= 2
    eye = np.full((C, C), -np.inf)
    np.fill_diagonal(eye, 0.0)
    nodes = [np.asarray(pot_b[t], np.float64) for t in range(E)] + [eye] * (P - E)
    while len(nodes) > 1:
        nxt = []
        for a, c in zip(nodes[0::2], nodes[1::2]):
            s = a[:, :, None] + c[None, :, :]           # [i, k, j]
            nxt.append(logsumexp(s, axis=1) if semiring == "log" else s.max(axis=1))
        nodes = nxt
    root = nodes[0]
    return logsumexp(root) if semiring == "log" else root.max()


@pytest.mark.parametrize("seed", range(3))
def test_tree_order_equals_sequential(seed):
    pot, lens = W.random_case(400 + seed, 4, 37, 5, lengths=[37, 20, 2, 1])
    z = oracle.logpartition(pot, lens)
    _, s = oracle.viterbi(pot, lens)
    for b in range(4):
        assert abs(_tree_logz(pot[b], lens[b], 5, "log") - z[b]) <= 1e-12 * max(1, abs(z[b]))
        assert _tree_logz(pot[b], lens[b], 5, "max") == s[b]     # exact in float64


# ----------------------------------------------------------------- sampled entry point
def test_marginals_seq_matches_full():
    pot, lens = W.random_case(9, 3, 12, 4, lengths=[12, 7, 1])
    z, m = oracle.marginals(pot, lens)
    for b in range(3):
        part, zb = oracle.marginals_seq(pot, lens, b, 2, 11)
        assert zb == z[b]
        np.testing.assert_array_equal(part, m[b, 2:11])


@pytest.mark.parametrize("B,N,C,lens", [(3, 12, 4, [12, 7, 1]), (2, 40, 9, [40, 2]),
                                        (4, 17, 1, None)])
def test_streamed_messages_match_full(B, N, C, lens):
    # the streamed entry points (messages once, then any range of edges) inherit every pin
    # of orc_marginals: they must reproduce its output bitwise, padding included
    pot, lens = W.random_case(10 + N, B, N, C, lengths=lens if lens is not None else "full")
    z, m = oracle.marginals(pot, lens)
    msg = oracle.Messages(pot, lens)
    np.testing.assert_array_equal(msg.logz, z)
    for b in range(B):
        for t0, t1 in ((0, N - 1), (0, 1), (N // 3, N - 1), (N - 2, N - 1)):
            if 0 <= t0 <= t1 <= N - 1:
                np.testing.assert_array_equal(msg.edge_marginals(b, t0, t1), m[b, t0:t1])
    with pytest.raises(ValueError):
        msg.edge_marginals(0, 0, N)          # past the last edge of the batch


def test_oracle_rejects_bad_lengths():
    pot = np.zeros((2, 3, 2, 2), np.float32)
    with pytest.raises(ValueError):
        oracle.logpartition(pot, np.array([5, 1], np.int32))
    with pytest.raises(ValueError):
        oracle.logpartition(pot, np.array([0, 1], np.int32))

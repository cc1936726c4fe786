"""GPU parity of the semi-Markov CRF (the chain scan over K*C expanded states) against the
float64 oracle's segmental forward-backward, on both chain paths (single launch for
K*C <= 32, multi-launch tree otherwise; TS_PATH=tree forces the tree).

Tolerances are the chain's: log Z and score 1e-5 relative (to max(|ref|, 1)), marginals
1e-5 absolute, labels and segment lengths bit-exact (the expanded chain's Viterbi sums are
float64 and exact, so its decisions are the oracle's; integer potentials force ties)."""
import numpy as np
import pytest

import oracle
from gpu_util import say
from paper_2002_00876_amd import workloads as W

pytestmark = pytest.mark.gpu

RTOL = 1e-5
ATOL = 1e-5


@pytest.fixture(params=["auto", "tree"], autouse=True)
def path_mode(request, monkeypatch):
    if request.param == "tree":
        monkeypatch.setenv("TS_PATH", "tree")
    else:
        monkeypatch.delenv("TS_PATH", raising=False)
    return request.param


def _gpu(sp, lens):
    import torch
    from paper_2002_00876_amd import binding
    dev = torch.device("cuda:0")
    tsp = torch.from_numpy(np.ascontiguousarray(sp)).to(dev)
    tl = torch.from_numpy(np.ascontiguousarray(lens)).to(dev)
    z = binding.semi_logpartition(tsp, tl)
    z2, m = binding.semi_marginals(tsp, tl)
    path, seglen, score = binding.semi_viterbi(tsp, tl)
    torch.cuda.synchronize()
    return [x.cpu().numpy() for x in (z, z2, m, path, seglen, score)]


def _rel(got, ref):
    fin = np.isfinite(ref)
    assert np.array_equal(np.isneginf(got), np.isneginf(ref)), "infinities differ"
    err = np.abs(got[fin].astype(np.float64) - ref[fin]) / np.maximum(np.abs(ref[fin]), 1.0)
    return err.max(initial=0.0)


def check_semi(sp, lens, tag):
    B, E, K, C, _ = sp.shape
    say(f"semi case {tag}: B={B} N={E + 1} K={K} C={C}")
    z, z2, m, path, seglen, score = _gpu(sp, lens)
    zo, mo = oracle.semi_marginals(sp, lens)
    po, go, so = oracle.semi_viterbi(sp, lens)
    assert _rel(z, zo) <= RTOL and _rel(z2, zo) <= RTOL, "log Z"
    for b in range(B):
        assert np.all(m[b, int(lens[b]) - 1:] == 0), "padding marginals are not exactly 0"
    err = np.abs(m.astype(np.float64) - mo).max(initial=0.0)
    assert err <= ATOL, f"marginals: max abs err {err:.3e}"
    fin = np.isfinite(so)
    assert np.array_equal(path[fin], po[fin]), "labels differ"
    assert np.array_equal(seglen[fin], go[fin]), "segment lengths differ"
    assert _rel(score, so) <= RTOL, "score"
    say(f"  ok: marginals max err {err:.2e}")


CASES = [
    # seed, B, N, K, C, kind
    (1, 4, 9, 2, 3, "normal"),
    (2, 5, 14, 3, 8, "normal"),      # K*C = 24: single launch
    (3, 3, 30, 4, 8, "int"),         # K*C = 32, exact ties
    (4, 4, 25, 5, 20, "normal"),     # K*C = 100: multi-launch tree
    (5, 3, 40, 6, 7, "int"),
    (6, 2, 12, 4, 64, "normal"),     # K*C = 256, the largest
    (7, 6, 33, 1, 20, "normal"),     # K = 1: the linear chain
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"seed{c[0]}-K{c[3]}-C{c[4]}")
def test_semi_random_cases(case):
    seed, B, N, K, C, kind = case
    sp, lens = W.semi_case(seed + 50, B, N, K, C, kind=kind)
    check_semi(sp, lens, f"seed {seed}")


def test_semi_forbidden_entries():
    sp, lens = W.semi_case(60, 5, 16, 3, 6, neg_inf_frac=0.4)
    check_semi(sp, lens, "-inf entries")


def test_semi_table1_shape():
    sp, lens = W.generate_semi("semi")
    check_semi(sp, lens, "Table 1 shape")


def test_semi_long_sampled():
    sp, lens = W.semi_case(61, 2, 300, 4, 32, len_range=(150, 300))
    check_semi(sp, lens, "long")


def test_k1_is_the_chain_bitwise():
    import torch
    from paper_2002_00876_amd import binding
    sp, lens = W.semi_case(62, 6, 30, 1, 20)
    dev = torch.device("cuda:0")
    tsp = torch.from_numpy(sp).to(dev)
    tl = torch.from_numpy(lens).to(dev)
    pot = tsp[:, :, 0].contiguous()
    z_s, m_s = binding.semi_marginals(tsp, tl)
    p_s, g_s, s_s = binding.semi_viterbi(tsp, tl)
    z_c, m_c = binding.marginals(pot, tl)
    p_c, s_c = binding.viterbi(pot, tl)
    assert torch.equal(z_s, z_c) and torch.equal(m_s[:, :, 0], m_c)
    assert torch.equal(p_s, p_c) and torch.equal(s_s, s_c)


def test_semi_single_token_batch():
    sp = np.zeros((3, 0, 4, 5, 5), np.float32)
    lens = np.ones(3, np.int32)
    z, z2, m, path, seglen, score = _gpu(sp, lens)
    np.testing.assert_allclose(z, np.log(5.0), rtol=1e-6)
    assert path.reshape(-1).tolist() == [0, 0, 0] and score.tolist() == [0.0] * 3

"""Parity of the HIP path (through the C ABI) with the float64 oracle: log Z within 1e-5
relative, marginals within 1e-5 absolute with padding exactly 0, Viterbi paths bit-exact
(lowest-index ties) and scores within 1e-5 relative."""
import numpy as np
import pytest

from gpu_util import check_all, check_logz, gpu_all, say
from paper_2002_00876_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(params=["auto", "tree"], autouse=True)
def path_mode(request, monkeypatch):
    """Run every case through the default dispatch (the fused single-launch kernels for
    C <= 32) and through the multi-launch tree forced by TS_PATH=tree."""
    if request.param == "tree":
        monkeypatch.setenv("TS_PATH", "tree")
    else:
        monkeypatch.delenv("TS_PATH", raising=False)
    return request.param


@pytest.mark.parametrize("name", ["tiny", "paper"])
def test_named_small_workloads(name):
    pot, lens = W.generate(name)
    check_all(pot, lens, name)


SHAPES = [  # (B, N, C): several tiles, ragged tails, odd label counts
    (3, 2, 5), (4, 3, 3), (5, 9, 20), (3, 17, 33), (2, 33, 64), (2, 24, 65),
    (2, 30, 128), (2, 12, 129), (1, 9, 256), (2, 7, 200), (3, 100, 16), (2, 257, 8),
    (4, 64, 1), (2, 5, 2), (3, 40, 31), (2, 18, 96),
    # every label padding of the single-launch kernels (C padded to 8, 16, 20, 24 or 32)
    (3, 13, 17), (2, 21, 19), (3, 11, 23), (2, 15, 24), (2, 9, 12), (3, 6, 28),
    # single-launch backtraces over several chunks of 32 edges: a last chunk of one edge, a
    # whole chunk, padded and unpadded multi-chunk sequences
    (3, 34, 7), (2, 33, 5), (3, 98, 8), (2, 161, 6),
    # the multi-launch outside sweep with each line split over 8 thread parts (32 labels)
    (2, 40, 32),
]


@pytest.mark.parametrize("B,N,C", SHAPES)
def test_random_shapes(B, N, C):
    lens = np.array(([1, 2, N] * B)[:B] if B >= 3 else [N, max(1, N // 2)][:B], np.int32)
    pot, lens = W.random_case(1000 + N * 7 + C, B, N, C, sigma=1.5, lengths=lens)
    check_all(pot, lens, f"random B={B} N={N} C={C}")


@pytest.mark.parametrize("B,N,C,r", [(4, 30, 5, 1), (3, 20, 20, 1), (2, 17, 64, 2), (2, 9, 130, 1),
                                     (3, 70, 4, 1)])
def test_integer_ties(B, N, C, r):
    pot, lens = W.random_case(2000 + C, B, N, C, kind="int", int_range=r, lengths="random")
    check_all(pot, lens, f"ties B={B} N={N} C={C}")


def test_neg_inf_entries():
    pot, lens = W.random_case(77, 4, 12, 6, lengths=[12, 9, 3, 1], neg_inf_frac=0.3)
    pot[1, 2] = -np.inf           # sequence 1 has no finite path
    check_all(pot, lens, "neg-inf")


def test_neg_inf_rows_and_columns_large_c():
    pot, lens = W.random_case(78, 2, 10, 70, lengths=[10, 7])
    pot[0, 3, 5, :] = -np.inf     # a label that cannot be left at edge 3
    pot[0, 4, :, 9] = -np.inf     # a label that cannot be entered at edge 4
    pot[1, 1, :, :40] = -np.inf
    check_all(pot, lens, "neg-inf rows/cols")


@pytest.mark.parametrize("C", [48, 20, 13])
def test_wide_dynamic_range_uses_exact_fallback(C):
    # sigma 40: exp-shifted products underflow and must be recomputed exactly (C = 20 and 13
    # take the single-launch kernels by default, C = 48 the multi-launch tree)
    pot, lens = W.random_case(79 + C, 3, 20, C, sigma=40.0, lengths=[20, 11, 2])
    check_all(pot, lens, f"sigma=40 C={C}")


def test_large_common_offset():
    pot, lens = W.random_case(80, 2, 40, 24, lengths=[40, 23])
    pot = (pot + np.float32(1000.0)).astype(np.float32)
    check_all(pot, lens, "offset 1000")


def test_single_token_batch():
    pot = np.zeros((3, 0, 4, 4), np.float32)
    lens = np.ones(3, np.int32)
    z, z2, m, path, score = gpu_all(pot, lens)
    np.testing.assert_allclose(z, np.log(4), rtol=1e-7)
    assert np.all(path == 0) and np.all(score == 0) and m.shape == (3, 0, 4, 4)


def test_no_lengths_means_full_length():
    import torch
    from paper_2002_00876_amd import binding
    import oracle
    pot, _ = W.random_case(81, 3, 20, 12, lengths="full")
    tp = torch.from_numpy(pot).cuda()
    z = binding.logpartition(tp, None).cpu().numpy()
    path, score = binding.viterbi(tp, None)
    check_logz(z, oracle.logpartition(pot, None))
    assert np.array_equal(path.cpu().numpy(), oracle.viterbi(pot, None)[0])


def test_bitwise_deterministic():
    pot, lens = W.generate("paper")
    a = gpu_all(pot, lens)
    b = gpu_all(pot, lens)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)

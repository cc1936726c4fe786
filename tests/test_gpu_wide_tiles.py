"""Parity of the multi-launch tree on shapes whose lower levels take the 128-wide output
tiles of the log-semiring product (a level uses them when it has at least 512 such tiles),
every marginal compared element by element: dense rows (C a multiple of 4, 16-byte loads)
and odd label counts (scalar loads), ragged lengths, exact integer ties and a wide dynamic
range."""
import numpy as np
import pytest

from gpu_util import check_all
from paper_2002_00876_amd import workloads as W

pytestmark = pytest.mark.gpu

CASES = [
    # (B, N, C, lengths): level 1 has B * 128 nodes, i.e. >= 512 tiles of 128 x 128
    (4, 257, 128, [257, 200, 131, 64]),
    (2, 129, 256, [129, 77]),
    (2, 257, 256, [257, 190]),
    (2, 257, 130, [257, 101]),    # two tiles per dimension, the second one ragged
    (3, 300, 192, [300, 299, 150]),
    (4, 257, 256, [257, 1, 2, 3]),    # sequences of one to three tokens beside a full one
]


@pytest.mark.parametrize("B,N,C,lens", CASES)
def test_wide_tiles_normal(B, N, C, lens):
    pot, lens = W.random_case(3000 + N + C, B, N, C, sigma=1.5, lengths=lens)
    check_all(pot, lens, f"wide tiles B={B} N={N} C={C}")


@pytest.mark.parametrize("B,N,C,lens", [CASES[0], CASES[3]])
def test_wide_tiles_integer_ties(B, N, C, lens):
    pot, lens = W.random_case(4000 + N + C, B, N, C, kind="int", int_range=1, lengths=lens)
    check_all(pot, lens, f"wide tiles, ties B={B} N={N} C={C}")


@pytest.mark.parametrize("B,N,C,lens", [(2, 600, 128, [600, 421]), (2, 200, 256, [200, 133])])
def test_wide_tiles_wide_dynamic_range(B, N, C, lens):
    # sigma 40 on shapes whose lower levels take the 128-wide full tiles (products from bf16
    # parts): those must keep float32 precision, and sums below 2^-80 take the exact
    # recomputation
    pot, lens = W.random_case(5000 + N + C, B, N, C, sigma=40.0, lengths=lens)
    check_all(pot, lens, f"wide tiles, sigma=40 B={B} N={N} C={C}")


def test_wide_tiles_product_underflow():
    # level-1 products on the 128-wide full tiles with entries whose shifted sum underflows
    # (S < 2^-80: every term below 2^-126) and takes the direct log-sum-exp: rows 5 and 77
    # of every even edge keep their mass on one contracted index, columns 9 and 200 of every
    # odd edge on another, so those entries of each level-1 product are about 2 e^-150 after
    # the shifts (the edges also reach magnitude 16: the float64 formation)
    B, N, C = 2, 257, 256
    pot, lens = W.random_case(6000, B, N, C, sigma=1.0, lengths=[257, 190])
    for t in range(0, N - 1, 2):
        for i, k0 in ((5, 3), (77, 100)):
            pot[:, t, i, :] -= 150.0
            pot[:, t, i, k0] += 150.0
    for t in range(1, N - 1, 2):
        for j, k1 in ((9, 50), (200, 201)):
            pot[:, t, :, j] -= 150.0
            pot[:, t, k1, j] += 150.0
    check_all(pot, lens, f"wide tiles, underflowing products B={B} N={N} C={C}")

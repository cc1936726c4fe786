"""Host-side checks of the C-ABI library: it loads, exports every entry point that
include/ts_chain.h declares, sizes workspaces, and rejects bad arguments with the
documented status codes before touching the device (no compute call is made here)."""
import ctypes
import os
import re

import pytest

from paper_2002_00876_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ts_chain.h")

FAKE = 0x10000          # 256-aligned, never dereferenced: every call below fails validation
TS_OK, NULL_ARG, BAD_DIM, WORKSPACE = 0, -1, -2, -3
# C = 40 takes the multi-launch tree, which needs a workspace; the fused path (C <= 32)
# needs none.  Every call here must fail validation before anything is launched.
CW = 40


@pytest.fixture(scope="module")
def L():
    return binding.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ts_[a-z_]+)\s*\(", text)))


def test_header_declares_the_three_calls():
    names = declared_functions()
    for n in ("ts_chain_logpartition", "ts_chain_marginals", "ts_chain_viterbi",
              "ts_chain_workspace_bytes", "ts_last_error", "ts_chain_max_labels"):
        assert n in names


def test_library_exports_every_declared_symbol(L):
    for name in declared_functions():
        assert hasattr(L, name), name
        assert ctypes.cast(getattr(L, name), ctypes.c_void_p).value


def test_max_labels(L):
    assert L.ts_chain_max_labels() == 256


def test_workspace_sizes(L, monkeypatch):
    ws = binding.workspace_bytes
    assert ws(0, 4, 1, 20) == 0 and ws(1, 4, 1, 20) == 0 and ws(2, 4, 1, 20) == 0
    for op in (0, 1, 2):
        assert ws(op, 32, 25, 20) == 0          # fused single-launch path: LDS only
        assert ws(op, 32, 25, CW) > 0
        assert ws(op, 32, 25, CW) % 256 == 0
        assert ws(op, 64, 25, CW) > ws(op, 32, 25, CW)
        assert ws(op, 32, 50, CW) > ws(op, 32, 25, CW)
    # marginals need the chunk nodes plus the outside vectors
    assert ws(1, 4, 513, CW) > ws(0, 4, 513, CW)
    # the tree over N-1 = 24 edges has levels of 16, 8, 4, 2, 1 nodes of C*C floats; with
    # at most 64 labels the chunk kernels fold chunks of 2^lc edges and run the recursions
    # over the chunk products, so only the chunk level is stored: for log Z lc follows the
    # length (4 edges for 24: 32 / 4 = 8 nodes), the marginals keep 16 edges (2 nodes)
    assert ws(0, 32, 25, CW) >= 32 * 8 * CW * CW * 4
    assert ws(0, 32, 25, CW) < 32 * (8 + 1) * CW * CW * 4
    assert 32 * 2 * CW * CW * 4 <= ws(1, 32, 25, CW) < 32 * 3 * CW * CW * 4
    # longer sequences take chunks of at most 16 edges: N - 1 = 512 edges, 32 chunk nodes
    node = CW * CW * 4 + 2 * CW * 8          # core and the float64 row and column offsets
    assert 4 * 32 * node <= ws(0, 4, 513, CW) < 4 * 32 * node + 4096
    # above 64 labels the marginals store every level; log Z with at most 128 labels stops
    # the up-sweep where the recursion over the level's nodes is cheaper than the levels
    # above it (here level 1: 16 nodes), above 128 labels it forms every level
    assert ws(1, 32, 25, 65) >= 32 * (16 + 8 + 4 + 2 + 1) * 65 * 65 * 4
    assert 32 * 16 * 65 * 65 * 4 <= ws(0, 32, 25, 65) < 32 * (16 + 8) * 65 * 65 * 4
    assert ws(0, 32, 25, 130) >= 32 * (16 + 8 + 4 + 2 + 1) * 130 * 130 * 4
    assert ws(7, 32, 25, CW) == 0 and ws(0, 0, 25, 20) == 0 and ws(0, 1, 25, 257) == 0
    assert ws(6, 32, 25, CW) >= ws(1, 32, 25, CW) + 32 * 24 * CW * CW * 4
    # entropy: the marginals workspace, the marginals themselves and per-edge partials;
    # log density: the log-partition workspace and log Z
    assert ws(4, 32, 25, CW) >= ws(1, 32, 25, CW) + 32 * 24 * CW * CW * 4 + 32 * 24 * 8
    assert ws(4, 32, 25, 20) >= 32 * 24 * 20 * 20 * 4
    assert ws(5, 32, 25, CW) >= ws(0, 32, 25, CW) + 32 * 4 and ws(5, 32, 25, 20) >= 32 * 4
    # the combined call: the marginals workspace followed by the Viterbi workspace
    assert ws(3, 32, 25, 20) == 0
    assert ws(3, 32, 25, CW) == ws(1, 32, 25, CW) + ws(2, 32, 25, CW)
    # TS_PATH=tree forces the multi-launch tree (with its chunk kernels) for small C too
    monkeypatch.setenv("TS_PATH", "tree")
    assert ws(0, 32, 25, 20) >= 32 * 2 * 20 * 20 * 4


def _err(L):
    return L.ts_last_error().decode()


def test_bad_dimensions_are_rejected(L):
    for B, N, C in [(0, 5, 3), (2, 0, 3), (2, 5, 0), (2, 5, 257), (-1, 5, 3)]:
        assert L.ts_chain_entropy(FAKE, None, B, N, C, FAKE, FAKE, 1 << 30, None) == BAD_DIM
        assert L.ts_chain_logpartition_sequential(FAKE, None, B, N, C, FAKE, None) == BAD_DIM
        assert L.ts_chain_sample(FAKE, None, FAKE, 1, B, N, C, FAKE, FAKE, 1 << 30, None) == BAD_DIM
        assert L.ts_chain_log_density(FAKE, None, FAKE, B, N, C, FAKE, FAKE, 1 << 30, None) == BAD_DIM
        assert L.ts_chain_logpartition(FAKE, None, B, N, C, FAKE, FAKE, 1 << 30, None) == BAD_DIM
        assert L.ts_chain_marginals(FAKE, None, B, N, C, FAKE, FAKE, FAKE, 1 << 30, None) == BAD_DIM
        assert L.ts_chain_viterbi(FAKE, None, B, N, C, FAKE, FAKE, FAKE, 1 << 30, None) == BAD_DIM
        assert L.ts_chain_marginals_viterbi(FAKE, None, B, N, C, FAKE, FAKE, FAKE, FAKE, FAKE,
                                            1 << 30, None) == BAD_DIM
    assert "ts_chain_max_labels" in _err(L) or "must" in _err(L)


def test_size_overflow_is_rejected(L):
    assert L.ts_chain_logpartition(FAKE, None, 1 << 40, 1 << 20, 256, FAKE, FAKE, 1, None) == BAD_DIM
    assert "overflow" in _err(L)
    # B * N beyond what one launch grid covers, even with tiny label sets
    assert L.ts_chain_logpartition(FAKE, None, 1 << 20, 1 << 10, 2, FAKE, FAKE, 1 << 40, None) == BAD_DIM
    assert L.ts_chain_workspace_bytes(0, 1 << 20, 1 << 10, 2) == 0
    assert L.ts_semimarkov_logpartition(FAKE, None, 1 << 20, 1 << 10, 1, 2, FAKE, FAKE, 1 << 40,
                                        None) == BAD_DIM
    # a huge label count with K = 1 is rejected before K * C is formed
    assert L.ts_semimarkov_logpartition(FAKE, None, 2, 5, 1, 1 << 62, FAKE, FAKE, 1 << 40,
                                        None) == BAD_DIM


def test_null_pointers_are_rejected(L):
    need = binding.workspace_bytes(0, 2, 5, CW)
    assert L.ts_chain_logpartition(None, None, 2, 5, CW, FAKE, FAKE, need, None) == NULL_ARG
    assert "pot" in _err(L)
    assert L.ts_chain_logpartition(FAKE, None, 2, 5, CW, None, FAKE, need, None) == NULL_ARG
    assert "logZ" in _err(L)
    assert L.ts_chain_logpartition(FAKE, None, 2, 5, CW, FAKE, None, need, None) == NULL_ARG
    assert "ws" in _err(L)
    need = binding.workspace_bytes(1, 2, 5, CW)
    assert L.ts_chain_marginals(FAKE, None, 2, 5, CW, FAKE, None, FAKE, need, None) == NULL_ARG
    assert "marg" in _err(L)
    need = binding.workspace_bytes(2, 2, 5, CW)
    assert L.ts_chain_viterbi(FAKE, None, 2, 5, CW, None, FAKE, FAKE, need, None) == NULL_ARG
    assert L.ts_chain_viterbi(FAKE, None, 2, 5, CW, FAKE, None, FAKE, need, None) == NULL_ARG
    need = binding.workspace_bytes(3, 2, 5, CW)
    mv = L.ts_chain_marginals_viterbi
    assert mv(None, None, 2, 5, CW, FAKE, FAKE, FAKE, FAKE, FAKE, need, None) == NULL_ARG
    assert mv(FAKE, None, 2, 5, CW, FAKE, None, FAKE, FAKE, FAKE, need, None) == NULL_ARG
    assert "marg" in _err(L)
    assert mv(FAKE, None, 2, 5, CW, FAKE, FAKE, None, FAKE, FAKE, need, None) == NULL_ARG
    assert mv(FAKE, None, 2, 5, CW, FAKE, FAKE, FAKE, None, FAKE, need, None) == NULL_ARG
    assert mv(FAKE, None, 2, 5, CW, FAKE, FAKE, FAKE, FAKE, None, need, None) == NULL_ARG
    assert "ws" in _err(L)
    assert mv(FAKE, None, 2, 5, CW, FAKE, FAKE, FAKE, FAKE, FAKE, need - 1, None) == WORKSPACE
    assert mv(FAKE, None, 2, 5, CW, FAKE, FAKE, FAKE, FAKE, FAKE + 16, need, None) == WORKSPACE
    assert mv(FAKE, None, 2, 5, 3, FAKE, FAKE, None, FAKE, None, 0, None) == NULL_ARG
    assert L.ts_chain_logpartition_sequential(FAKE, None, 2, 5, CW, None, None) == NULL_ARG
    need = binding.workspace_bytes(6, 2, 5, CW)
    assert L.ts_chain_sample(FAKE, None, FAKE, 0, 2, 5, CW, FAKE, FAKE, need, None) == BAD_DIM
    assert L.ts_chain_sample(FAKE, None, None, 3, 2, 5, CW, FAKE, FAKE, need, None) == NULL_ARG
    assert L.ts_chain_sample(FAKE, None, FAKE, 3, 2, 5, CW, None, FAKE, need, None) == NULL_ARG
    assert L.ts_chain_sample(FAKE, None, FAKE, 3, 2, 5, CW, FAKE, FAKE, need - 1, None) == WORKSPACE
    assert L.ts_chain_logpartition_sequential(None, None, 2, 5, CW, FAKE, None) == NULL_ARG
    need = binding.workspace_bytes(4, 2, 5, CW)
    assert L.ts_chain_entropy(FAKE, None, 2, 5, CW, None, FAKE, need, None) == NULL_ARG
    assert "entropy" in _err(L)
    assert L.ts_chain_entropy(FAKE, None, 2, 5, CW, FAKE, FAKE, need - 1, None) == WORKSPACE
    assert L.ts_chain_entropy(None, None, 2, 5, CW, FAKE, FAKE, need, None) == NULL_ARG
    need = binding.workspace_bytes(5, 2, 5, CW)
    assert L.ts_chain_log_density(FAKE, None, None, 2, 5, CW, FAKE, FAKE, need, None) == NULL_ARG
    assert L.ts_chain_log_density(FAKE, None, FAKE, 2, 5, CW, None, FAKE, need, None) == NULL_ARG
    assert L.ts_chain_log_density(FAKE, None, FAKE, 2, 5, CW, FAKE, FAKE + 16, need, None) == WORKSPACE
    # the fused path (no workspace) still rejects missing outputs
    assert L.ts_chain_marginals(FAKE, None, 2, 5, 3, FAKE, None, None, 0, None) == NULL_ARG
    assert L.ts_chain_viterbi(FAKE, None, 2, 5, 3, None, FAKE, None, 0, None) == NULL_ARG


def test_small_or_misaligned_workspace_is_rejected(L):
    for op, fn in ((0, "logpartition"), (1, "marginals"), (2, "viterbi")):
        need = binding.workspace_bytes(op, 4, 9, CW)
        f = getattr(L, "ts_chain_" + fn)
        args = {0: (FAKE,), 1: (FAKE, FAKE), 2: (FAKE, FAKE)}[op]
        assert f(FAKE, None, 4, 9, CW, *args, FAKE, need - 1, None) == WORKSPACE
        assert "workspace too small" in _err(L)
        assert f(FAKE, None, 4, 9, CW, *args, FAKE + 16, need, None) == WORKSPACE
        assert "aligned" in _err(L)


def test_semimarkov_workspace_sizes(L):
    sw = binding.semi_workspace_bytes
    # expanded edges [B, N-1, KC, KC] come first, then the chain plan over K*C labels
    B, N, K, C = 32, 25, 5, 20
    x = B * (N - 1) * (K * C) ** 2 * 4
    assert sw(0, B, N, K, C) >= x + binding.workspace_bytes(0, B, N, K * C)
    assert sw(1, B, N, K, C) >= 2 * x + binding.workspace_bytes(1, B, N, K * C)
    assert sw(2, B, N, K, C) >= x + B * N * 4 + binding.workspace_bytes(2, B, N, K * C)
    assert all(sw(op, B, N, K, C) % 256 == 0 for op in (0, 1, 2))
    # small expanded label sets keep the chain on its single-launch path
    assert sw(0, B, N, 2, 8) == B * (N - 1) * 16 * 16 * 4
    assert sw(0, 4, 1, 5, 20) == 0                    # one token: no edges
    assert sw(3, B, N, K, C) == 0 and sw(0, B, N, 0, C) == 0
    assert sw(0, B, N, 13, 20) == 0                   # K * C = 260 > 256


def test_semimarkov_bad_arguments_are_rejected(L):
    for B, N, K, C in [(0, 5, 2, 3), (2, 0, 2, 3), (2, 5, 0, 3), (2, 5, 2, 0), (2, 5, 13, 20)]:
        assert L.ts_semimarkov_logpartition(FAKE, None, B, N, K, C, FAKE, FAKE, 1 << 30,
                                            None) == BAD_DIM
        assert L.ts_semimarkov_marginals(FAKE, None, B, N, K, C, FAKE, FAKE, FAKE, 1 << 30,
                                         None) == BAD_DIM
        assert L.ts_semimarkov_viterbi(FAKE, None, B, N, K, C, FAKE, FAKE, FAKE, FAKE, 1 << 30,
                                       None) == BAD_DIM
    B, N, K, C = 2, 5, 3, 20
    need = binding.semi_workspace_bytes(0, B, N, K, C)
    assert L.ts_semimarkov_logpartition(None, None, B, N, K, C, FAKE, FAKE, need, None) == NULL_ARG
    assert "sp" in _err(L)
    assert L.ts_semimarkov_logpartition(FAKE, None, B, N, K, C, None, FAKE, need, None) == NULL_ARG
    assert L.ts_semimarkov_logpartition(FAKE, None, B, N, K, C, FAKE, FAKE, need - 1,
                                        None) == WORKSPACE
    assert L.ts_semimarkov_logpartition(FAKE, None, B, N, K, C, FAKE, FAKE + 16, need,
                                        None) == WORKSPACE
    need = binding.semi_workspace_bytes(1, B, N, K, C)
    assert L.ts_semimarkov_marginals(FAKE, None, B, N, K, C, FAKE, None, FAKE, need,
                                     None) == NULL_ARG
    assert L.ts_semimarkov_marginals(FAKE, None, B, N, K, C, FAKE, FAKE, None, need,
                                     None) == NULL_ARG
    need = binding.semi_workspace_bytes(2, B, N, K, C)
    vit = L.ts_semimarkov_viterbi
    assert vit(FAKE, None, B, N, K, C, None, FAKE, FAKE, FAKE, need, None) == NULL_ARG
    assert vit(FAKE, None, B, N, K, C, FAKE, None, FAKE, FAKE, need, None) == NULL_ARG
    assert vit(FAKE, None, B, N, K, C, FAKE, FAKE, None, FAKE, need, None) == NULL_ARG
    assert vit(FAKE, None, B, N, K, C, FAKE, FAKE, FAKE, FAKE, need - 1, None) == WORKSPACE


def test_viterbi_decode_length_limit_is_rejected(L):
    # the backtrace tables must fit in LDS: with C = 256 at most 65536 edges per sequence.
    # The marginals plan alone accepts this size; the combined call must still refuse it
    # (before any device call) as ts_chain_viterbi does.
    B, N, C = 1, 70000, 256
    assert binding.workspace_bytes(1, B, N, C) > 0
    assert binding.workspace_bytes(2, B, N, C) == 0
    assert binding.workspace_bytes(3, B, N, C) == 0
    big = 1 << 40
    assert L.ts_chain_viterbi(FAKE, None, B, N, C, FAKE, FAKE, FAKE, big, None) == BAD_DIM
    assert L.ts_chain_marginals_viterbi(FAKE, None, B, N, C, FAKE, FAKE, FAKE, FAKE, FAKE, big,
                                        None) == BAD_DIM
    assert "overflow" in _err(L) or "range" in _err(L)
    # the largest accepted length at C = 256 (65536 edges)
    assert binding.workspace_bytes(2, 1, 65537, C) > 0
    assert binding.workspace_bytes(2, 1, 65538, C) == 0


def test_noalloc_entry_point_rejects_oversized_problems(L):
    # the allocation-free marginals call checks the workspace it would need against its
    # fixed per-GPU scratch before any device call
    cap = L.ts_chain_noalloc_scratch_bytes()
    assert cap == 64 << 20
    B, N, C = 4, 400, 128
    assert binding.workspace_bytes(1, B, N, C) > cap
    assert L.ts_chain_marginals_noalloc(FAKE, None, B, N, C, FAKE, FAKE, None) == BAD_DIM
    assert "scratch" in _err(L)
    # the call's own argument checks still apply
    assert L.ts_chain_marginals_noalloc(FAKE, None, 0, 5, 3, FAKE, FAKE, None) == BAD_DIM

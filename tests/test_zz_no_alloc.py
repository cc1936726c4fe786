"""The allocation-free marginals entry point (ts_chain_marginals_noalloc, per-GPU scratch
array inside the library) against ts_chain_marginals with a caller workspace: two calls in
a row on the same scratch, the second on a smaller problem, each compared with the
workspace call (same kernels: bitwise equal) and with the float64 oracle to the hot path's
bar (log Z 1e-5 relative, marginals 1e-5 absolute, padding exactly 0)."""
import numpy as np
import pytest

from gpu_util import check_logz, check_marg, say
from paper_2002_00876_amd import workloads as W

pytestmark = pytest.mark.gpu


def _case(B, N, C, seed, lens):
    import torch

    import oracle
    from paper_2002_00876_amd import binding

    pot, lens = W.random_case(seed, B, N, C, sigma=1.5, lengths=lens)
    assert binding.workspace_bytes(binding.OP_MARGINALS, B, N, C) <= binding.noalloc_scratch_bytes()
    tp = torch.from_numpy(pot).cuda()
    tl = torch.from_numpy(lens).cuda()
    say(f"noalloc case B={B} N={N} C={C}")
    z1, m1 = binding.marginals(tp, tl)
    z2, m2 = binding.marginals_noalloc(tp, tl)
    torch.cuda.synchronize()
    assert torch.equal(z1, z2), "log Z differs from the workspace call"
    assert torch.equal(m1, m2), "marginals differ from the workspace call"
    zo, mo = oracle.marginals(pot, lens)
    check_logz(z2.cpu().numpy(), zo)
    check_marg(m2.cpu().numpy(), mo, lens)


def test_noalloc_two_calls_second_smaller():
    # multi-launch tree (workspace-backed kernels): full 128-wide tiles first, then a
    # smaller problem with an odd label count reusing the same scratch
    _case(2, 129, 128, 9001, [129, 70])
    _case(3, 60, 40, 9002, [60, 31, 1])


def test_noalloc_single_launch_path_needs_no_scratch():
    # small label sets take the single-launch kernels, which use LDS only
    _case(4, 25, 20, 9003, [25, 13, 2, 1])


def test_noalloc_rejects_problems_beyond_the_scratch():
    import torch

    from paper_2002_00876_amd import binding

    B, N, C = 4, 400, 128
    assert binding.workspace_bytes(binding.OP_MARGINALS, B, N, C) > binding.noalloc_scratch_bytes()
    tp = torch.zeros((B, N - 1, C, C), dtype=torch.float32, device="cuda")
    with pytest.raises(binding.TsError) as ei:
        binding.marginals_noalloc(tp)
    assert ei.value.code == -2 and "scratch" in str(ei.value)

"""The boundary's optional validation (environment variable TS_CHECK=1): lengths outside
[1, N] give TS_ERR_LENGTHS and labels outside [0, C) give TS_ERR_LABELS, from a host-side
check made before anything is launched; valid inputs give the same outputs as without the
check."""
import numpy as np
import pytest

from paper_2002_00876_amd import workloads as W

pytestmark = pytest.mark.gpu

ERR_LENGTHS, ERR_LABELS = -4, -6


def _tensors(dev, pot_h, lens_h):
    import torch
    return torch.from_numpy(pot_h).to(dev), torch.from_numpy(np.asarray(lens_h, np.int32)).to(dev)


@pytest.mark.parametrize("C", [20, 64, 128])
@pytest.mark.parametrize("bad", [0, -3, 41])
def test_bad_lengths_rejected(C, bad, monkeypatch):
    import torch
    from paper_2002_00876_amd import binding
    monkeypatch.setenv("TS_CHECK", "1")
    dev = torch.device("cuda:0")
    pot_h, _ = W.random_case(31, 3, 40, C)
    pot, lens = _tensors(dev, pot_h, [40, bad, 7])
    calls = [lambda: binding.logpartition(pot, lens), lambda: binding.marginals(pot, lens),
             lambda: binding.viterbi(pot, lens), lambda: binding.marginals_viterbi(pot, lens),
             lambda: binding.entropy(pot, lens)]
    for call in calls:
        with pytest.raises(binding.TsError) as ei:
            call()
        assert ei.value.code == ERR_LENGTHS
    torch.cuda.synchronize()


@pytest.mark.parametrize("bad", [-1, 20])
def test_bad_labels_rejected(bad, monkeypatch):
    import torch
    from paper_2002_00876_amd import binding
    monkeypatch.setenv("TS_CHECK", "1")
    dev = torch.device("cuda:0")
    pot_h, lens_h = W.random_case(32, 3, 12, 20, lengths=[12, 5, 1])
    pot, lens = _tensors(dev, pot_h, lens_h)
    labels = np.zeros((3, 12), np.int32)
    labels[1, 4] = bad                      # inside sequence 1 (length 5)
    with pytest.raises(binding.TsError) as ei:
        binding.log_density(pot, torch.from_numpy(labels).to(dev), lens)
    assert ei.value.code == ERR_LABELS
    labels[1, 4] = 0
    labels[1, 7] = bad                      # past the end of sequence 1: not checked
    binding.log_density(pot, torch.from_numpy(labels).to(dev), lens)
    torch.cuda.synchronize()


@pytest.mark.parametrize("C", [20, 64, 128])
def test_valid_inputs_unchanged_by_the_check(C, monkeypatch):
    import torch
    from paper_2002_00876_amd import binding
    dev = torch.device("cuda:0")
    pot_h, lens_h = W.random_case(33, 4, 70, C, lengths=[70, 1, 33, 69])
    pot, lens = _tensors(dev, pot_h, lens_h)
    plain = [t.cpu() for t in binding.marginals_viterbi(pot, lens)]
    monkeypatch.setenv("TS_CHECK", "1")
    checked = [t.cpu() for t in binding.marginals_viterbi(pot, lens)]
    for a, b, name in zip(plain, checked, ("logZ", "marginals", "path", "score")):
        assert torch.equal(a, b), f"{name} differs with TS_CHECK=1"

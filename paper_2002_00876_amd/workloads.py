"""Seeded synthetic workloads shaped like the paper's linear-chain benchmarks.

This module only draws inputs; it contains none of the inference arithmetic, so the
GPU path and the CPU oracle can both be fed from it.  Every workload is an edge
log-potential tensor ``pot`` of shape [B, N-1, C, C] in float32 plus int32 token
lengths [B] (1 <= len <= N).

Recipe (identical for every consumer):
  * ``rng = numpy.random.default_rng(seed)``;
  * potentials are drawn first, one sequence at a time (``rng.standard_normal((N-1, C, C))``
    for b = 0..B-1), scaled by sigma in float64, then cast to float32 once;
  * lengths are drawn afterwards with ``rng.integers(lo, hi, endpoint=True, size=B)``
    unless the workload fixes them;
  * the HMM-style workload draws a shared transition matrix T ~ N(0,1) [C, C] and
    emissions e ~ N(0,1) [B, N, C], then sets
    pot[b,t,i,j] = log_softmax_j(T)[i,j] + e[b,t,j] in float64 and casts to float32.

The five named workloads follow the batch/length/label shapes of the paper's
linear-chain timing (batch 32, N=25, C=20, Table 1) and of longer, wider chains.
"""
from dataclasses import dataclass
from typing import Optional, Tuple

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    N: int
    C: int
    seed: int
    kind: str = "normal"          # "normal" or "hmm"
    sigma: float = 1.0
    len_range: Optional[Tuple[int, int]] = None   # inclusive; None -> all N
    fixed_lengths: Optional[Tuple[int, ...]] = None

    @property
    def shape(self):
        return (self.B, self.N - 1, self.C, self.C)

    def describe(self):
        return {"workload": self.name, "B": self.B, "N": self.N, "C": self.C}


WORKLOADS = {
    "tiny": Workload("tiny", 2, 6, 3, seed=1),
    "paper": Workload("paper", 32, 25, 20, seed=2, len_range=(13, 25)),
    "mid": Workload("mid", 32, 512, 64, seed=3, sigma=2.0, len_range=(256, 512)),
    "hmm": Workload("hmm", 16, 1024, 256, seed=4, kind="hmm"),
    "long": Workload("long", 4, 8192, 128, seed=5, fixed_lengths=(8192, 6000, 4096, 1024)),
}

# the same five, in order: tiny, paper-shaped, mid, HMM-style, long
ORDER = ("tiny", "paper", "mid", "hmm", "long")


def _log_softmax_rows(T):
    m = T.max(axis=1, keepdims=True)
    z = T - m
    return z - np.log(np.exp(z).sum(axis=1, keepdims=True))


def generate(w, out=None):
    """Materialise workload ``w`` (a Workload or its name) -> (pot float32, lengths int32).

    ``out`` may be a preallocated float32 array of shape w.shape (e.g. a pinned buffer's
    numpy view) to avoid a second copy of large inputs.
    """
    if isinstance(w, str):
        w = WORKLOADS[w]
    B, N, C = w.B, w.N, w.C
    E = N - 1
    rng = np.random.default_rng(w.seed)
    pot = out if out is not None else np.empty((B, E, C, C), np.float32)
    assert pot.shape == (B, E, C, C) and pot.dtype == np.float32
    if w.kind == "normal":
        for b in range(B):
            x = rng.standard_normal((E, C, C))
            if w.sigma != 1.0:
                x *= w.sigma
            pot[b] = x
    elif w.kind == "hmm":
        T = rng.standard_normal((C, C))
        e = rng.standard_normal((B, N, C))
        lsm = _log_softmax_rows(T)
        tmp = np.empty((E, C, C), np.float64)
        for b in range(B):
            np.add(lsm[None, :, :], e[b, :E, None, :], out=tmp)
            pot[b] = tmp
    else:
        raise ValueError(w.kind)
    if w.fixed_lengths is not None:
        lengths = np.asarray(w.fixed_lengths, np.int32)
    elif w.len_range is not None:
        lo, hi = w.len_range
        lengths = rng.integers(lo, hi, endpoint=True, size=B).astype(np.int32)
    else:
        lengths = np.full(B, N, np.int32)
    return pot, lengths


def random_case(seed, B, N, C, kind="normal", sigma=1.0, lengths="random", int_range=2,
                neg_inf_frac=0.0):
    """Small seeded cases for tests.

    kind: "normal" (sigma * N(0,1)), "int" (uniform integers in [-int_range, int_range],
    which forces exact ties), "zero".  lengths: "random" (uniform in [1, N]), "full",
    or an explicit sequence.  neg_inf_frac sets that fraction of entries to -inf.
    """
    rng = np.random.default_rng(seed)
    E = N - 1
    if kind == "normal":
        pot = (rng.standard_normal((B, E, C, C)) * sigma).astype(np.float32)
    elif kind == "int":
        pot = rng.integers(-int_range, int_range, endpoint=True,
                           size=(B, E, C, C)).astype(np.float32)
    elif kind == "zero":
        pot = np.zeros((B, E, C, C), np.float32)
    else:
        raise ValueError(kind)
    if neg_inf_frac > 0:
        mask = rng.random((B, E, C, C)) < neg_inf_frac
        pot[mask] = -np.inf
    if isinstance(lengths, str):
        if lengths == "random":
            lens = rng.integers(1, N, endpoint=True, size=B)
        elif lengths == "full":
            lens = np.full(B, N)
        else:
            raise ValueError(lengths)
    else:
        lens = np.asarray(lengths)
    return pot, lens.astype(np.int32)


# Semi-Markov CRF: segment potentials sp [B, N-1, K, C, C] (Table 1's timing shape for the
# semi-Markov row: batch 32, N=25, C=20, K=5).  Same recipe: potentials first, one sequence
# at a time (rng.standard_normal((N-1, K, C, C))), scaled by sigma in float64 and cast to
# float32 once, then lengths.
SEMI_WORKLOADS = {
    "semi": dict(B=32, N=25, K=5, C=20, seed=6, len_range=(13, 25)),
    "semi_long": dict(B=8, N=1024, K=8, C=32, seed=7, len_range=(512, 1024)),
}


def semi_case(seed, B, N, K, C, sigma=1.0, len_range=None, kind="normal", int_range=1,
              neg_inf_frac=0.0):
    """Seeded semi-Markov segment potentials [B, N-1, K, C, C] (float32) and lengths [B].
    kind "int" draws integers in [-int_range, int_range] (exact ties); len_range None gives
    lengths uniform in [1, N]."""
    rng = np.random.default_rng(seed)
    shape = (N - 1, K, C, C)
    if kind == "normal":
        sp = np.stack([rng.standard_normal(shape) * sigma for _ in range(B)])
    elif kind == "int":
        sp = np.stack([rng.integers(-int_range, int_range, endpoint=True, size=shape)
                       for _ in range(B)]).astype(np.float64)
    else:
        raise ValueError(kind)
    if neg_inf_frac > 0:
        sp[rng.random(sp.shape) < neg_inf_frac] = -np.inf
    lo, hi = len_range if len_range is not None else (1, N)
    lengths = rng.integers(lo, hi, endpoint=True, size=B).astype(np.int32)
    return sp.astype(np.float32), lengths


def generate_semi(name):
    w = SEMI_WORKLOADS[name]
    return semi_case(w["seed"], w["B"], w["N"], w["K"], w["C"], len_range=w["len_range"])

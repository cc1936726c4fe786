"""Brute-force enumeration of every label sequence of tiny linear-chain CRFs.

Independent of the oracle: it scores each of the C**L sequences directly from the
CRF definition (Torch-Struct Sec. 5.1: p(z) = exp(z.l) / sum_z' exp(z'.l), parts are
the labelled edges of Sec. 5.2) and reads every quantity off that list:
  log Z            = log sum_z exp score(z)
  mu[t,i,j]        = sum over z with z_t=i, z_{t+1}=j of p(z)
  A*               = max_z score(z)
  canonical argmax = among the max-score sequences, the smallest under the key
                     (z_{L-1}, z_{L-2}, ..., z_0) -- the sequence a backtrace that
                     always takes the lowest index produces.
  entropy          = -sum_z p(z) log p(z)
  log p(z)         = score(z) - log Z   (brute_log_density)
"""
import itertools
import math

import numpy as np


def enumerate_seq(pot_b, L, C):
    """All (z, score) pairs for one sequence with L tokens; pot_b is [N-1, C, C]."""
    out = []
    for z in itertools.product(range(C), repeat=L):
        s = 0.0
        for t in range(L - 1):
            s += float(pot_b[t, z[t], z[t + 1]])
        out.append((z, s))
    return out


def brute(pot, lengths):
    """-> logZ [B], mu [B, N-1, C, C], score [B], path [B, N] (all float64 / int32)."""
    pot = np.asarray(pot, dtype=np.float64)
    B, E, C, _ = pot.shape
    N = E + 1
    logZ = np.zeros(B)
    mu = np.zeros((B, E, C, C))
    score = np.zeros(B)
    path = np.full((B, N), -1, np.int32)
    for b in range(B):
        L = int(lengths[b])
        seqs = enumerate_seq(pot[b], L, C)
        scores = [s for _, s in seqs]
        m = max(scores)
        if m == -math.inf:
            logZ[b] = -math.inf
        else:
            logZ[b] = m + math.log(sum(math.exp(s - m) for s in scores))
            for z, s in seqs:
                p = math.exp(s - logZ[b])
                for t in range(L - 1):
                    mu[b, t, z[t], z[t + 1]] += p
        score[b] = m
        best = [z for z, s in seqs if s == m]
        zb = min(best, key=lambda z: tuple(reversed(z)))
        path[b, :L] = zb
    return logZ, mu, score, path


def brute_entropy(pot, lengths):
    """-> H [B] = -sum_z p(z) log p(z) by enumeration (0 when no sequence is finite)."""
    pot = np.asarray(pot, dtype=np.float64)
    B, E, C, _ = pot.shape
    H = np.zeros(B)
    for b in range(B):
        seqs = enumerate_seq(pot[b], int(lengths[b]), C)
        scores = [s for _, s in seqs]
        m = max(scores)
        if m == -math.inf:
            continue
        lz = m + math.log(sum(math.exp(s - m) for s in scores))
        h = 0.0
        for s in scores:
            if s != -math.inf:
                p = math.exp(s - lz)
                h -= p * (s - lz)
        H[b] = h
    return H


def brute_log_density(pot, lengths, labels):
    """-> log p(z_b) [B] for the given label sequences, from the enumerated log Z."""
    pot = np.asarray(pot, dtype=np.float64)
    B, E, C, _ = pot.shape
    out = np.zeros(B)
    for b in range(B):
        L = int(lengths[b])
        scores = [s for _, s in enumerate_seq(pot[b], L, C)]
        m = max(scores)
        lz = m + math.log(sum(math.exp(s - m) for s in scores))
        z = labels[b]
        out[b] = sum(float(pot[b, t, z[t], z[t + 1]]) for t in range(L - 1)) - lz
    return out

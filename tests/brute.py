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


def compositions(E, K):
    """All ordered tuples of segment lengths in 1..K that sum to E."""
    if E == 0:
        yield ()
        return
    for k in range(1, min(K, E) + 1):
        for rest in compositions(E - k, K):
            yield (k,) + rest


def enumerate_segmentations(sp_b, E, K, C):
    """All labelled segmentations of E steps for one sequence, sp_b [N-1, K, C, C]: a list
    of (starts, lengths, labels y_0..y_m, score) with score = sum_m sp[s_m, k_m-1, y_{m-1}, y_m]
    (Table 1's semi-Markov parts: a segment's potential depends on its start, its length,
    its label and the previous segment's label; y_0 is a free initial label)."""
    out = []
    for ks in compositions(E, K):
        starts = [sum(ks[:m]) for m in range(len(ks))]
        for ys in itertools.product(range(C), repeat=len(ks) + 1):
            s = 0.0
            for m, (t, k) in enumerate(zip(starts, ks)):
                s += float(sp_b[t, k - 1, ys[m], ys[m + 1]])
            out.append((starts, ks, ys, s))
    return out


def brute_semi(sp, lengths):
    """Semi-Markov CRF by enumeration -> logZ [B], mu [B, N-1, K, C, C], score [B],
    path [B, N], seglen [B, N-1].  The canonical argmax is the max-score segmentation that
    is smallest under the key (y_m, k_m, y_{m-1}, k_{m-1}, ..., k_1, y_0): the one a
    backtrace produces that always takes the last label lowest, then the shortest last
    segment, then the lowest previous label."""
    sp = np.asarray(sp, dtype=np.float64)
    B, E1, K, C, _ = sp.shape
    N = E1 + 1
    logZ = np.zeros(B)
    mu = np.zeros((B, E1, K, C, C))
    score = np.zeros(B)
    path = np.full((B, N), -1, np.int32)
    seglen = np.full((B, E1), -1, np.int32)
    for b in range(B):
        E = int(lengths[b]) - 1
        segs = enumerate_segmentations(sp[b], E, K, C)
        scores = [s for *_, s in segs]
        m = max(scores)
        if E == 0:
            logZ[b] = math.log(C)
        elif m == -math.inf:
            logZ[b] = -math.inf
        else:
            logZ[b] = m + math.log(sum(math.exp(s - m) for s in scores))
            for starts, ks, ys, s in segs:
                p = math.exp(s - logZ[b])
                for mm, (t, k) in enumerate(zip(starts, ks)):
                    mu[b, t, k - 1, ys[mm], ys[mm + 1]] += p
        score[b] = m

        def key(seg):
            starts, ks, ys, _ = seg
            out = []
            for mm in range(len(ks), 0, -1):
                out += [ys[mm], ks[mm - 1]]
            return tuple(out + [ys[0]])

        starts, ks, ys, _ = min((g for g in segs if g[3] == m), key=key)
        path[b, 0] = ys[0]
        seglen[b, :E] = 0
        for mm, (t, k) in enumerate(zip(starts, ks)):
            path[b, t + 1:t + k + 1] = ys[mm + 1]
            seglen[b, t] = k
    return logZ, mu, score, path, seglen

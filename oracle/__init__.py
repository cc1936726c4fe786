"""Float64 CPU oracle for batched linear-chain (and semi-Markov) CRF inference.

TEST INFRASTRUCTURE ONLY: the slow, plain checker the HIP path is compared against.
Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import it.  The product package never does.

The arithmetic lives in ``oracle.c`` (sequential forward-backward and Viterbi DP in
float64, following Torch-Struct Sec. 5.1-5.2); this module only marshals numpy arrays
through ctypes.  Build with ``build()`` (gcc, no fast-math).
"""
import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None


def compile_source(src, lib):
    """gcc -O2 -fopenmp (no fast-math) of one oracle source file into a shared library."""
    tmp = lib + ".tmp"
    subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11",
                           "-Wall", "-Wextra", src, "-o", tmp, "-lm"])
    os.replace(tmp, lib)
    return lib


def build(force=True):
    """Compile oracle.c into liboracle.so."""
    if not force and os.path.exists(_LIB):
        return _LIB
    return compile_source(_SRC, _LIB)


def load_library(path):
    """Load a compiled oracle library (the default one, or a test's variant of it)."""
    lib = ctypes.CDLL(path)
    i64, p = ctypes.c_int64, ctypes.c_void_p
    for name in ("orc_logpartition", "orc_logpartition_f64"):
        getattr(lib, name).argtypes = [p, p, i64, i64, i64, p]
    for name in ("orc_marginals", "orc_marginals_f64"):
        getattr(lib, name).argtypes = [p, p, i64, i64, i64, p, p]
    for name in ("orc_viterbi", "orc_viterbi_f64"):
        getattr(lib, name).argtypes = [p, p, i64, i64, i64, p, p]
    lib.orc_marginals_seq.argtypes = [p, p, i64, i64, i64, i64, i64, i64, p, p]
    if hasattr(lib, "orc_messages"):
        lib.orc_messages.argtypes = [p, p, i64, i64, i64, p, p, p]
        lib.orc_edge_marginals.argtypes = [p, p, i64, i64, i64, p, p, p, i64, i64, i64, p]
    if hasattr(lib, "orc_entropy"):
        lib.orc_entropy.argtypes = [p, p, i64, i64, i64, p]
        lib.orc_log_density.argtypes = [p, p, p, i64, i64, i64, p]
        lib.orc_sample.argtypes = [p, p, p, i64, i64, i64, i64, p, p]
    if hasattr(lib, "orc_semi_marginals"):
        for name in ("orc_semi_marginals", "orc_semi_marginals_f64"):
            getattr(lib, name).argtypes = [p, p, i64, i64, i64, i64, p, p]
        lib.orc_semi_viterbi.argtypes = [p, p, i64, i64, i64, i64, p, p, p]
    lib.orc_max_threads.restype = ctypes.c_int
    return lib


def _load(lib=None):
    global _lib
    if lib is not None:
        return lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        _lib = load_library(_LIB)
    return _lib


def _prep(pot, lengths):
    pot = np.asarray(pot)
    if pot.ndim != 4 or pot.shape[2] != pot.shape[3]:
        raise ValueError("potentials must be [B, N-1, C, C]")
    if pot.dtype == np.float64:
        pot = np.ascontiguousarray(pot)
        f64 = True
    else:
        pot = np.ascontiguousarray(pot, dtype=np.float32)
        f64 = False
    B, E, C, _ = pot.shape
    N = E + 1
    if lengths is not None:
        lengths = np.ascontiguousarray(lengths, dtype=np.int32)
        if lengths.shape != (B,):
            raise ValueError("lengths must be [B]")
    return pot, lengths, f64, B, N, C


def _ptr(a):
    return None if a is None else a.ctypes.data


def _check(rc):
    if rc != 0:
        raise ValueError(f"oracle rejected its arguments (code {rc})")


def logpartition(pot, lengths=None, lib=None):
    """log Z[b] (float64 [B]) for potentials [B, N-1, C, C] and token lengths [B]."""
    pot, lengths, f64, B, N, C = _prep(pot, lengths)
    out = np.empty(B, np.float64)
    fn = _load(lib).orc_logpartition_f64 if f64 else _load(lib).orc_logpartition
    _check(fn(_ptr(pot), _ptr(lengths), B, N, C, _ptr(out)))
    return out


def marginals(pot, lengths=None, lib=None):
    """(log Z [B], edge marginals [B, N-1, C, C]) in float64."""
    pot, lengths, f64, B, N, C = _prep(pot, lengths)
    logz = np.empty(B, np.float64)
    marg = np.empty((B, max(N - 1, 0), C, C), np.float64)
    fn = _load(lib).orc_marginals_f64 if f64 else _load(lib).orc_marginals
    _check(fn(_ptr(pot), _ptr(lengths), B, N, C, _ptr(logz), _ptr(marg)))
    return logz, marg


def viterbi(pot, lengths=None, lib=None):
    """(path int32 [B, N], -1 past each length; score float64 [B])."""
    pot, lengths, f64, B, N, C = _prep(pot, lengths)
    path = np.empty((B, N), np.int32)
    score = np.empty(B, np.float64)
    fn = _load(lib).orc_viterbi_f64 if f64 else _load(lib).orc_viterbi
    _check(fn(_ptr(pot), _ptr(lengths), B, N, C, _ptr(path), _ptr(score)))
    return path, score


def entropy(pot, lengths=None, lib=None):
    """Entropy H[b] (float64 [B]) of each sequence's label distribution (fp32 potentials)."""
    pot, lengths, f64, B, N, C = _prep(pot, lengths)
    if f64:
        raise ValueError("entropy takes fp32 potentials")
    out = np.empty(B, np.float64)
    _check(_load(lib).orc_entropy(_ptr(pot), _ptr(lengths), B, N, C, _ptr(out)))
    return out


def log_density(pot, labels, lengths=None, lib=None):
    """log p(z_b) (float64 [B]) of label sequences labels [B, N] (int, entries past each
    length ignored) under fp32 potentials."""
    pot, lengths, f64, B, N, C = _prep(pot, lengths)
    if f64:
        raise ValueError("log_density takes fp32 potentials")
    labels = np.ascontiguousarray(labels, dtype=np.int32)
    if labels.shape != (B, N):
        raise ValueError("labels must be [B, N]")
    out = np.empty(B, np.float64)
    _check(_load(lib).orc_log_density(_ptr(pot), _ptr(lengths), _ptr(labels), B, N, C, _ptr(out)))
    return out


def sample(pot, uniforms, lengths=None, lib=None):
    """Forward-filtering backward-sampling draws with the given uniforms [S, B, N] in
    [0, 1): (paths int32 [S, B, N] with -1 past each length, margin float64 [S, B] -- the
    closest any draw of that sequence came to picking a neighbouring label, relative to the
    draw's total weight)."""
    pot, lengths, f64, B, N, C = _prep(pot, lengths)
    if f64:
        raise ValueError("sample takes fp32 potentials")
    uniforms = np.ascontiguousarray(uniforms, dtype=np.float32)
    if uniforms.ndim != 3 or uniforms.shape[1:] != (B, N):
        raise ValueError("uniforms must be [S, B, N]")
    S = uniforms.shape[0]
    paths = np.empty((S, B, N), np.int32)
    margin = np.empty((S, B), np.float64)
    _check(_load(lib).orc_sample(_ptr(pot), _ptr(lengths), _ptr(uniforms), S, B, N, C,
                                 _ptr(paths), _ptr(margin)))
    return paths, margin


def marginals_seq(pot, lengths, b, t0, t1):
    """Marginals of edges [t0, t1) of sequence b only (fp32 potentials), and log Z[b]."""
    pot, lengths, f64, B, N, C = _prep(pot, lengths)
    if f64:
        raise ValueError("marginals_seq takes fp32 potentials")
    out = np.empty((t1 - t0, C, C), np.float64)
    logz = ctypes.c_double()
    _check(_load().orc_marginals_seq(_ptr(pot), _ptr(lengths), B, N, C, b, t0, t1, _ptr(out),
                                     ctypes.addressof(logz)))
    return out, logz.value


class Messages:
    """Forward and backward log-messages of every sequence (one pass of the recursions),
    from which the marginals of any range of edges can be formed in bounded memory."""

    def __init__(self, pot, lengths=None, lib=None):
        pot, lengths, f64, B, N, C = _prep(pot, lengths)
        if f64:
            raise ValueError("Messages takes fp32 potentials")
        self._lib = _load(lib)
        self.pot, self.lengths, self.B, self.N, self.C = pot, lengths, B, N, C
        self.alpha = np.empty((B, N, C), np.float64)
        self.beta = np.empty((B, N, C), np.float64)
        self.logz = np.empty(B, np.float64)
        _check(self._lib.orc_messages(_ptr(pot), _ptr(lengths), B, N, C, _ptr(self.alpha),
                                      _ptr(self.beta), _ptr(self.logz)))

    def edge_marginals(self, b, t0, t1, out=None):
        """Marginals of edges [t0, t1) of sequence b, float64 [(t1-t0), C, C] (0 for
        padding edges); bitwise equal to the same slice of marginals()."""
        C = self.C
        if out is None:
            out = np.empty((t1 - t0, C, C), np.float64)
        assert out.dtype == np.float64 and out.flags.c_contiguous and out.shape == (t1 - t0, C, C)
        _check(self._lib.orc_edge_marginals(_ptr(self.pot), _ptr(self.lengths), self.B, self.N,
                                            C, _ptr(self.alpha), _ptr(self.beta),
                                            _ptr(self.logz), b, t0, t1, _ptr(out)))
        return out


def max_threads():
    """OpenMP threads available to the oracle's parallel loops."""
    return _load().orc_max_threads()


def _prep_semi(sp, lengths):
    sp = np.asarray(sp)
    if sp.ndim != 5 or sp.shape[3] != sp.shape[4]:
        raise ValueError("semi-Markov potentials must be [B, N-1, K, C, C]")
    f64 = sp.dtype == np.float64
    sp = np.ascontiguousarray(sp, dtype=np.float64 if f64 else np.float32)
    B, E, K, C, _ = sp.shape
    if lengths is not None:
        lengths = np.ascontiguousarray(lengths, dtype=np.int32)
        if lengths.shape != (B,):
            raise ValueError("lengths must be [B]")
    return sp, lengths, f64, B, E + 1, K, C


def semi_marginals(sp, lengths=None, lib=None):
    """Semi-Markov CRF: (log Z [B], segment marginals [B, N-1, K, C, C]) in float64, for
    segment potentials sp [B, N-1, K, C, C]: sp[b, t, k-1, i, j] scores a segment of length
    k starting at step t with label j after a segment labelled i."""
    sp, lengths, f64, B, N, K, C = _prep_semi(sp, lengths)
    logz = np.empty(B, np.float64)
    marg = np.empty((B, N - 1, K, C, C), np.float64)
    fn = _load(lib).orc_semi_marginals_f64 if f64 else _load(lib).orc_semi_marginals
    _check(fn(_ptr(sp), _ptr(lengths), B, N, K, C, _ptr(logz), _ptr(marg)))
    return logz, marg


def semi_logpartition(sp, lengths=None, lib=None):
    """Semi-Markov CRF log Z [B] (float64)."""
    sp, lengths, f64, B, N, K, C = _prep_semi(sp, lengths)
    logz = np.empty(B, np.float64)
    fn = _load(lib).orc_semi_marginals_f64 if f64 else _load(lib).orc_semi_marginals
    _check(fn(_ptr(sp), _ptr(lengths), B, N, K, C, _ptr(logz), None))
    return logz


def semi_viterbi(sp, lengths=None, lib=None):
    """Semi-Markov CRF best segmentation: (path int32 [B, N] -- path[0] the free initial
    label, path[t+1] the label of the segment covering step t; seglen int32 [B, N-1] -- the
    length of the segment starting at step t, else 0; both -1 past each sequence; score
    float64 [B])."""
    sp, lengths, f64, B, N, K, C = _prep_semi(sp, lengths)
    if f64:
        raise ValueError("semi_viterbi takes fp32 potentials")
    path = np.empty((B, N), np.int32)
    seglen = np.empty((B, N - 1), np.int32)
    score = np.empty(B, np.float64)
    _check(_load(lib).orc_semi_viterbi(_ptr(sp), _ptr(lengths), B, N, K, C, _ptr(path),
                                       _ptr(seglen), _ptr(score)))
    return path, seglen, score

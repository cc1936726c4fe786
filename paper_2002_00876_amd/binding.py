"""Python binding of libtschain.so: marshals torch tensors (device memory and the
current HIP stream) into the C ABI of include/ts_chain.h.  No arithmetic happens here;
every step runs in the library's HIP kernels.  If the library is missing, every call
raises: there is no fallback."""
import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libtschain.so")

OP_LOGPARTITION, OP_MARGINALS, OP_VITERBI, OP_MARGINALS_VITERBI = 0, 1, 2, 3
OP_ENTROPY, OP_LOG_DENSITY, OP_SAMPLE = 4, 5, 6
STATUS = {0: "TS_OK", -1: "TS_ERR_NULL_ARG", -2: "TS_ERR_BAD_DIM", -3: "TS_ERR_WORKSPACE",
          -4: "TS_ERR_LENGTHS", -5: "TS_ERR_HIP", -6: "TS_ERR_LABELS"}

_lib = None


class TsError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{STATUS.get(code, code)}: {msg}")
        self.code = code


def lib():
    """The loaded C library with argument types declared (raises if it was not built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: run paper_2002_00876_amd.build.build()")
        L = ctypes.CDLL(LIB_PATH)
        i64, p, sz = ctypes.c_int64, ctypes.c_void_p, ctypes.c_size_t
        L.ts_chain_max_labels.restype = ctypes.c_int
        L.ts_chain_workspace_bytes.argtypes = [ctypes.c_int, i64, i64, i64]
        L.ts_chain_workspace_bytes.restype = sz
        L.ts_chain_logpartition.argtypes = [p, p, i64, i64, i64, p, p, sz, p]
        L.ts_chain_marginals.argtypes = [p, p, i64, i64, i64, p, p, p, sz, p]
        L.ts_chain_viterbi.argtypes = [p, p, i64, i64, i64, p, p, p, sz, p]
        L.ts_chain_marginals_viterbi.argtypes = [p, p, i64, i64, i64, p, p, p, p, p, sz, p]
        L.ts_chain_marginals_noalloc.argtypes = [p, p, i64, i64, i64, p, p, p]
        L.ts_chain_noalloc_scratch_bytes.restype = sz
        L.ts_chain_entropy.argtypes = [p, p, i64, i64, i64, p, p, sz, p]
        L.ts_chain_log_density.argtypes = [p, p, p, i64, i64, i64, p, p, sz, p]
        L.ts_chain_logpartition_sequential.argtypes = [p, p, i64, i64, i64, p, p]
        L.ts_chain_sample.argtypes = [p, p, p, i64, i64, i64, i64, p, p, sz, p]
        L.ts_semimarkov_workspace_bytes.argtypes = [ctypes.c_int, i64, i64, i64, i64]
        L.ts_semimarkov_workspace_bytes.restype = sz
        L.ts_semimarkov_logpartition.argtypes = [p, p, i64, i64, i64, i64, p, p, sz, p]
        L.ts_semimarkov_marginals.argtypes = [p, p, i64, i64, i64, i64, p, p, p, sz, p]
        L.ts_semimarkov_viterbi.argtypes = [p, p, i64, i64, i64, i64, p, p, p, p, sz, p]
        for f in ("ts_chain_logpartition", "ts_chain_marginals", "ts_chain_viterbi",
                  "ts_chain_marginals_noalloc",
                  "ts_chain_marginals_viterbi", "ts_chain_entropy", "ts_chain_log_density",
                  "ts_chain_logpartition_sequential", "ts_chain_sample",
                  "ts_semimarkov_logpartition", "ts_semimarkov_marginals",
                  "ts_semimarkov_viterbi"):
            getattr(L, f).restype = ctypes.c_int
        L.ts_last_error.restype = ctypes.c_char_p
        _lib = L
    return _lib


def _check(code):
    if code != 0:
        raise TsError(code, lib().ts_last_error().decode())


def _ptr(t):
    return None if t is None else t.data_ptr()


def _stream(device):
    return torch.cuda.current_stream(device).cuda_stream


def _prep(pot, lengths):
    if not pot.is_cuda:
        raise ValueError("pot must be a device tensor")
    if pot.dtype != torch.float32 or pot.dim() != 4 or pot.shape[2] != pot.shape[3]:
        raise ValueError("pot must be float32 [B, N-1, C, C]")
    pot = pot.contiguous()
    B, E, C, _ = pot.shape
    if lengths is not None:
        if lengths.device != pot.device or lengths.dtype != torch.int32 or lengths.shape != (B,):
            raise ValueError("lengths must be int32 [B] on the same device as pot")
        lengths = lengths.contiguous()
    return pot, lengths, B, E + 1, C


def workspace_bytes(op, B, N, C):
    return lib().ts_chain_workspace_bytes(op, B, N, C)


def _workspace(op, B, N, C, device, ws=None):
    need = workspace_bytes(op, B, N, C)
    if ws is not None:
        return ws, ws.numel() * ws.element_size()
    if need == 0:
        return None, 0
    return torch.empty(need, dtype=torch.uint8, device=device), need


def logpartition(pot, lengths=None, out=None, ws=None):
    """log Z [B] (float32) of potentials [B, N-1, C, C] with token lengths [B]."""
    pot, lengths, B, N, C = _prep(pot, lengths)
    logz = out if out is not None else torch.empty(B, dtype=torch.float32, device=pot.device)
    w, nb = _workspace(OP_LOGPARTITION, B, N, C, pot.device, ws)
    _check(lib().ts_chain_logpartition(_ptr(pot), _ptr(lengths), B, N, C, _ptr(logz), _ptr(w),
                                       nb, _stream(pot.device)))
    return logz


def marginals(pot, lengths=None, out=None, ws=None, want_logz=True):
    """(log Z [B] or None, edge marginals [B, N-1, C, C]), float32."""
    pot, lengths, B, N, C = _prep(pot, lengths)
    if out is not None:
        logz, marg = out
    else:
        logz = torch.empty(B, dtype=torch.float32, device=pot.device) if want_logz else None
        marg = torch.empty_like(pot)
    w, nb = _workspace(OP_MARGINALS, B, N, C, pot.device, ws)
    _check(lib().ts_chain_marginals(_ptr(pot), _ptr(lengths), B, N, C, _ptr(logz),
                                    _ptr(marg) if N > 1 else None, _ptr(w), nb,
                                    _stream(pot.device)))
    return logz, marg


def noalloc_scratch_bytes():
    """Bytes of the per-GPU scratch array of the allocation-free marginals call."""
    return lib().ts_chain_noalloc_scratch_bytes()


def marginals_noalloc(pot, lengths=None, out=None, want_logz=True):
    """marginals() through ts_chain_marginals_noalloc: no workspace; the library's per-GPU
    scratch array is used instead (calls on one GPU must not overlap)."""
    pot, lengths, B, N, C = _prep(pot, lengths)
    if out is not None:
        logz, marg = out
    else:
        logz = torch.empty(B, dtype=torch.float32, device=pot.device) if want_logz else None
        marg = torch.empty_like(pot)
    _check(lib().ts_chain_marginals_noalloc(_ptr(pot), _ptr(lengths), B, N, C, _ptr(logz),
                                            _ptr(marg) if N > 1 else None,
                                            _stream(pot.device)))
    return logz, marg


def viterbi(pot, lengths=None, out=None, ws=None):
    """(path int32 [B, N] with -1 past each length, score float32 [B])."""
    pot, lengths, B, N, C = _prep(pot, lengths)
    if out is not None:
        path, score = out
    else:
        path = torch.empty((B, N), dtype=torch.int32, device=pot.device)
        score = torch.empty(B, dtype=torch.float32, device=pot.device)
    w, nb = _workspace(OP_VITERBI, B, N, C, pot.device, ws)
    _check(lib().ts_chain_viterbi(_ptr(pot), _ptr(lengths), B, N, C, _ptr(path), _ptr(score),
                                  _ptr(w), nb, _stream(pot.device)))
    return path, score


def marginals_viterbi(pot, lengths=None, out=None, ws=None, want_logz=True):
    """(log Z [B] or None, marginals [B, N-1, C, C], path [B, N], score [B]) in one call."""
    pot, lengths, B, N, C = _prep(pot, lengths)
    if out is not None:
        logz, marg, path, score = out
    else:
        dev = pot.device
        logz = torch.empty(B, dtype=torch.float32, device=dev) if want_logz else None
        marg = torch.empty_like(pot)
        path = torch.empty((B, N), dtype=torch.int32, device=dev)
        score = torch.empty(B, dtype=torch.float32, device=dev)
    w, nb = _workspace(OP_MARGINALS_VITERBI, B, N, C, pot.device, ws)
    _check(lib().ts_chain_marginals_viterbi(_ptr(pot), _ptr(lengths), B, N, C, _ptr(logz),
                                            _ptr(marg) if N > 1 else None, _ptr(path),
                                            _ptr(score), _ptr(w), nb, _stream(pot.device)))
    return logz, marg, path, score


def entropy(pot, lengths=None, out=None, ws=None):
    """Entropy [B] (float32) of each sequence's label distribution."""
    pot, lengths, B, N, C = _prep(pot, lengths)
    h = out if out is not None else torch.empty(B, dtype=torch.float32, device=pot.device)
    w, nb = _workspace(OP_ENTROPY, B, N, C, pot.device, ws)
    _check(lib().ts_chain_entropy(_ptr(pot), _ptr(lengths), B, N, C, _ptr(h), _ptr(w), nb,
                                  _stream(pot.device)))
    return h


def log_density(pot, labels, lengths=None, out=None, ws=None):
    """log p(z) [B] (float32) of label sequences labels (int32 [B, N])."""
    pot, lengths, B, N, C = _prep(pot, lengths)
    if labels.device != pot.device or labels.dtype != torch.int32 or labels.shape != (B, N):
        raise ValueError("labels must be int32 [B, N] on the same device as pot")
    labels = labels.contiguous()
    lp = out if out is not None else torch.empty(B, dtype=torch.float32, device=pot.device)
    w, nb = _workspace(OP_LOG_DENSITY, B, N, C, pot.device, ws)
    _check(lib().ts_chain_log_density(_ptr(pot), _ptr(lengths), _ptr(labels), B, N, C, _ptr(lp),
                                      _ptr(w), nb, _stream(pot.device)))
    return lp


def logpartition_sequential(pot, lengths=None, out=None):
    """log Z [B] by the left-to-right forward algorithm (the serial baseline of the scan)."""
    pot, lengths, B, N, C = _prep(pot, lengths)
    logz = out if out is not None else torch.empty(B, dtype=torch.float32, device=pot.device)
    _check(lib().ts_chain_logpartition_sequential(_ptr(pot), _ptr(lengths), B, N, C, _ptr(logz),
                                                  _stream(pot.device)))
    return logz


def sample(pot, uniforms, lengths=None, out=None, ws=None):
    """Forward-filtering backward-sampling draws: paths int32 [S, B, N] (-1 past each
    length) from caller-supplied uniforms float32 [S, B, N] in [0, 1)."""
    pot, lengths, B, N, C = _prep(pot, lengths)
    if (uniforms.device != pot.device or uniforms.dtype != torch.float32 or uniforms.dim() != 3
            or tuple(uniforms.shape[1:]) != (B, N)):
        raise ValueError("uniforms must be float32 [S, B, N] on the same device as pot")
    uniforms = uniforms.contiguous()
    S = uniforms.shape[0]
    paths = out if out is not None else torch.empty((S, B, N), dtype=torch.int32,
                                                    device=pot.device)
    w, nb = _workspace(OP_SAMPLE, B, N, C, pot.device, ws)
    _check(lib().ts_chain_sample(_ptr(pot), _ptr(lengths), _ptr(uniforms), S, B, N, C,
                                 _ptr(paths), _ptr(w), nb, _stream(pot.device)))
    return paths


# ---- semi-Markov CRF: segment potentials sp [B, N-1, K, C, C] ----

def _prep_semi(sp, lengths):
    if not sp.is_cuda:
        raise ValueError("sp must be a device tensor")
    if sp.dtype != torch.float32 or sp.dim() != 5 or sp.shape[3] != sp.shape[4]:
        raise ValueError("sp must be float32 [B, N-1, K, C, C]")
    sp = sp.contiguous()
    B, E, K, C, _ = sp.shape
    if lengths is not None:
        if lengths.device != sp.device or lengths.dtype != torch.int32 or lengths.shape != (B,):
            raise ValueError("lengths must be int32 [B] on the same device as sp")
        lengths = lengths.contiguous()
    return sp, lengths, B, E + 1, K, C


def semi_workspace_bytes(op, B, N, K, C):
    return lib().ts_semimarkov_workspace_bytes(op, B, N, K, C)


def _semi_workspace(op, B, N, K, C, device, ws=None):
    if ws is not None:
        return ws, ws.numel() * ws.element_size()
    need = semi_workspace_bytes(op, B, N, K, C)
    if need == 0:
        return None, 0
    return torch.empty(need, dtype=torch.uint8, device=device), need


def semi_logpartition(sp, lengths=None, out=None, ws=None):
    """Semi-Markov log Z [B] (float32)."""
    sp, lengths, B, N, K, C = _prep_semi(sp, lengths)
    logz = out if out is not None else torch.empty(B, dtype=torch.float32, device=sp.device)
    w, nb = _semi_workspace(OP_LOGPARTITION, B, N, K, C, sp.device, ws)
    _check(lib().ts_semimarkov_logpartition(_ptr(sp), _ptr(lengths), B, N, K, C, _ptr(logz),
                                            _ptr(w), nb, _stream(sp.device)))
    return logz


def semi_marginals(sp, lengths=None, out=None, ws=None, want_logz=True):
    """Semi-Markov (log Z [B] or None, segment marginals [B, N-1, K, C, C]), float32."""
    sp, lengths, B, N, K, C = _prep_semi(sp, lengths)
    if out is not None:
        logz, marg = out
    else:
        logz = torch.empty(B, dtype=torch.float32, device=sp.device) if want_logz else None
        marg = torch.empty_like(sp)
    w, nb = _semi_workspace(OP_MARGINALS, B, N, K, C, sp.device, ws)
    _check(lib().ts_semimarkov_marginals(_ptr(sp), _ptr(lengths), B, N, K, C, _ptr(logz),
                                         _ptr(marg) if N > 1 else None, _ptr(w), nb,
                                         _stream(sp.device)))
    return logz, marg


def semi_viterbi(sp, lengths=None, out=None, ws=None):
    """Semi-Markov best segmentation: (path int32 [B, N], seglen int32 [B, N-1],
    score float32 [B])."""
    sp, lengths, B, N, K, C = _prep_semi(sp, lengths)
    if out is not None:
        path, seglen, score = out
    else:
        dev = sp.device
        path = torch.empty((B, N), dtype=torch.int32, device=dev)
        seglen = torch.empty((B, N - 1), dtype=torch.int32, device=dev)
        score = torch.empty(B, dtype=torch.float32, device=dev)
    w, nb = _semi_workspace(OP_VITERBI, B, N, K, C, sp.device, ws)
    _check(lib().ts_semimarkov_viterbi(_ptr(sp), _ptr(lengths), B, N, K, C, _ptr(path),
                                       _ptr(seglen) if N > 1 else None, _ptr(score), _ptr(w),
                                       nb, _stream(sp.device)))
    return path, seglen, score

"""Fastmax fp64 CPU oracle -- test infrastructure only.

A plain, slow, obviously-correct float64 implementation of Fastmax attention
(arXiv 2402.07901, Sec. 2.2 definition, Sec. 2.4 factorisation, Sec. 2.3 score
derivative), written in C (``fastmax_ref.c``) and wrapped here with ctypes.

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s CPU-baseline
leg may import this package.  The HIP library never calls it, and the two
share no code.  Inputs are float64 numpy arrays in [B, H, N, D] layout.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "fastmax_ref.c")
_LIB_DEFAULT = os.path.join(_HERE, "libfastmax_oracle.so")
# the sanitizer tier (tests/test_sanitize.py) points this at the
# AddressSanitizer/UBSan build of the same source
_LIB = os.environ.get("FASTMAX_ORACLE_LIB", _LIB_DEFAULT)
LIB_ASAN = os.path.join(_HERE, "libfastmax_oracle_asan.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2, OpenMP). Returns the library path."""
    if force or not os.path.exists(_LIB_DEFAULT):
        tmp = _LIB_DEFAULT + ".tmp"
        cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
               "-Wall", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_DEFAULT)
    return _LIB_DEFAULT


def build_sanitized() -> str:
    """Compile the oracle with AddressSanitizer and UndefinedBehaviorSanitizer
    (gcc; any report aborts).  Returns the library path; a process loading it
    needs gcc's libasan preloaded."""
    tmp = LIB_ASAN + ".tmp"
    cmd = ["gcc", "-O1", "-g", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-Wall",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-fno-omit-frame-pointer", "-o", tmp, _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB_ASAN)
    return LIB_ASAN


def _bind(path):
    """Load a compiled oracle library and declare its signatures."""
    lib = ctypes.CDLL(path)
    dp = ctypes.POINTER(ctypes.c_double)
    L = ctypes.c_long
    I = ctypes.c_int
    lib.fmo_num_threads.restype = I
    lib.fmo_standardize.argtypes = [dp, L, L, dp, dp, dp]
    F = ctypes.c_double
    lib.fmo_attention_matrix.argtypes = [dp, dp, L, L, I, I, F, dp]
    lib.fmo_fwd_brute.argtypes = [dp, dp, dp, L, L, L, L, I, I, F, dp, dp, dp]
    lib.fmo_fwd_fact.argtypes = [dp, dp, dp, L, L, L, L, I, I, F, dp, dp]
    lib.fmo_fwd_rows.argtypes = [dp, dp, dp, L, L, L, L, I, I, F, L,
                                 ctypes.POINTER(ctypes.c_int64), dp, dp, dp]
    lib.fmo_bwd_brute.argtypes = [dp, dp, dp, dp, dp, L, L, L, L, I, I, F,
                                  dp, dp, dp]
    up = ctypes.POINTER(ctypes.c_uint32)
    lib.fmo_mask_words.argtypes = [L]
    lib.fmo_mask_words.restype = L
    lib.fmo_philox4x32_10.argtypes = [up, up, up]
    lib.fmo_dropout_mask.argtypes = [L, L, L, L, F, ctypes.c_uint64, up]
    lib.fmo_fwd_drop_brute.argtypes = [dp, dp, dp, up, L, L, L, L, I, F, F, dp, dp]
    lib.fmo_fwd_drop_fact.argtypes = [dp, dp, dp, up, L, L, L, L, I, F, F, dp, dp]
    lib.fmo_bwd_drop_brute.argtypes = [dp, dp, dp, dp, dp, up, L, L, L, L, I, F, F,
                                       dp, dp, dp]
    return lib


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        _lib = _bind(_LIB)
    return _lib


def _f64(x):
    return np.ascontiguousarray(x, dtype=np.float64)


def _ptr(a):
    if a is None:
        return None
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _shape4(q):
    if q.ndim != 4:
        raise ValueError("expected [B, H, N, D]")
    return q.shape


def num_threads() -> int:
    """OpenMP threads the oracle uses."""
    return int(_load().fmo_num_threads())


def standardize(x):
    """Eqs. (6)-(7): per-row (q - mean) / population std over the last axis.

    Returns (xhat, mean, std) with mean/std shaped like x without its last axis.
    """
    x = _f64(x)
    D = x.shape[-1]
    rows = x.size // D
    xh = np.empty_like(x)
    mu = np.empty(x.shape[:-1])
    sg = np.empty(x.shape[:-1])
    _load().fmo_standardize(_ptr(x), rows, D, _ptr(xh), _ptr(mu), _ptr(sg))
    return xh, mu, sg


def attention_matrix(q, k, p, causal, scale=1.0):
    """Explicit N x N Fastmax attention matrix of ONE head, q/k shaped [N, D];
    weights f_p(scale * q^.k^)."""
    q, k = _f64(q), _f64(k)
    N, D = q.shape
    A = np.empty((N, N))
    _load().fmo_attention_matrix(_ptr(q), _ptr(k), N, D, int(p), int(causal),
                                 float(scale), _ptr(A))
    return A


def fwd_brute(q, k, v, p, causal, with_abs=False, scale=1.0):
    """Brute force O(N^2 D) forward with weights f_p(scale * s); returns
    (O, G) or, with ``with_abs``, (O, G, sum_n |w_in|)."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    B, H, N, D = _shape4(q)
    out = np.empty_like(q)
    g = np.empty((B, H, N))
    gabs = np.empty((B, H, N)) if with_abs else None
    _load().fmo_fwd_brute(_ptr(q), _ptr(k), _ptr(v), B, H, N, D, int(p),
                          int(causal), float(scale), _ptr(out), _ptr(g), _ptr(gabs))
    return (out, g, gabs) if with_abs else (out, g)


def fwd_fact(q, k, v, p, causal, scale=1.0):
    """Factorised moment forward (Sec. 2.4) with weights f_p(scale * s);
    returns (O, G)."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    B, H, N, D = _shape4(q)
    out = np.empty_like(q)
    g = np.empty((B, H, N))
    _load().fmo_fwd_fact(_ptr(q), _ptr(k), _ptr(v), B, H, N, D, int(p),
                         int(causal), float(scale), _ptr(out), _ptr(g))
    return out, g


def fwd_rows(q, k, v, p, causal, rows, with_abs=False, scale=1.0):
    """Brute force for selected rows (flat index b*H*N + h*N + i).

    Returns (O_rows [n, D], G_rows [n]) and, with ``with_abs``, also
    sum_n |w_in| per row.
    """
    q, k, v = _f64(q), _f64(k), _f64(v)
    B, H, N, D = _shape4(q)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    out = np.empty((rows.size, D))
    g = np.empty(rows.size)
    gabs = np.empty(rows.size) if with_abs else None
    _load().fmo_fwd_rows(_ptr(q), _ptr(k), _ptr(v), B, H, N, D, int(p),
                         int(causal), float(scale), rows.size,
                         rows.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
                         _ptr(out), _ptr(g), _ptr(gabs))
    return (out, g, gabs) if with_abs else (out, g)


def bwd_brute(q, k, v, dout, p, causal, o_used=None, scale=1.0):
    """Brute force O(N^2 D) backward; returns (dq, dk, dv).

    ``o_used``: the forward output the gradient is taken at (default: the
    exact O).  Tests pass the oracle's own O rounded to the I/O dtype to model
    a backward that consumes the stored output."""
    q, k, v, dout = _f64(q), _f64(k), _f64(v), _f64(dout)
    B, H, N, D = _shape4(q)
    if o_used is not None:
        o_used = _f64(o_used)
        assert o_used.shape == q.shape
    dq = np.empty_like(q)
    dk = np.empty_like(q)
    dv = np.empty_like(q)
    _load().fmo_bwd_brute(_ptr(q), _ptr(k), _ptr(v), _ptr(dout), _ptr(o_used),
                          B, H, N, D, int(p), int(causal), float(scale), _ptr(dq),
                          _ptr(dk), _ptr(dv))
    return dq, dk, dv


# ---------------------------------------------------------------------------
# "Quadratic" dropout (Sec. 2.4, dropout paragraph; Fig. 2): keep bits on each
# key token's D(D+1)/2 quadratic features, kept ones scaled by 1/(1 - rate).
# ``bits`` is uint32 [B, H, N, mask_words(D)]; feature t(m, l) = m D -
# m(m-1)/2 + l - m (m <= l) is bit t % 32 of word t // 32.
# ---------------------------------------------------------------------------
def _uptr(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32))


def mask_words(D):
    """uint32 words per token of a keep-bit row: ceil(D(D+1)/2 / 32)."""
    return int(_load().fmo_mask_words(int(D)))


def philox4x32_10(ctr, key):
    """Philox4x32-10 (Salmon et al., SC 2011): 4 counter words, 2 key words
    -> 4 output words."""
    c = np.ascontiguousarray(ctr, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    o = np.empty(4, dtype=np.uint32)
    _load().fmo_philox4x32_10(_uptr(c), _uptr(k), _uptr(o))
    return o


def dropout_mask(B, H, N, D, rate, seed):
    """Keep bits drawn with Philox4x32-10: key = (seed & 0xffffffff, seed >> 32),
    counter = (n, t // 4, b H + h, 0), word t % 4; dropped iff the word is below
    floor(rate 2^32)."""
    bits = np.empty((B, H, N, mask_words(D)), dtype=np.uint32)
    _load().fmo_dropout_mask(B, H, N, D, float(rate), ctypes.c_uint64(int(seed)), _uptr(bits))
    return bits


def _bits(bits, B, H, N, D):
    b = np.ascontiguousarray(bits, dtype=np.uint32)
    if b.shape != (B, H, N, mask_words(D)):
        raise ValueError(f"keep bits shaped {b.shape}, expected {(B, H, N, mask_words(D))}")
    return b


def fwd_drop_brute(q, k, v, bits, rate, causal, scale=1.0):
    """Brute force forward (p = 2) with the masked weights; returns (O, G)."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    B, H, N, D = _shape4(q)
    b = _bits(bits, B, H, N, D)
    out = np.empty_like(q)
    g = np.empty((B, H, N))
    _load().fmo_fwd_drop_brute(_ptr(q), _ptr(k), _ptr(v), _uptr(b), B, H, N, D, int(causal),
                               float(scale), float(rate), _ptr(out), _ptr(g))
    return out, g


def fwd_drop_fact(q, k, v, bits, rate, causal, scale=1.0):
    """Factorised forward (p = 2) with the masked quadratic embedding; (O, G)."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    B, H, N, D = _shape4(q)
    b = _bits(bits, B, H, N, D)
    out = np.empty_like(q)
    g = np.empty((B, H, N))
    _load().fmo_fwd_drop_fact(_ptr(q), _ptr(k), _ptr(v), _uptr(b), B, H, N, D, int(causal),
                              float(scale), float(rate), _ptr(out), _ptr(g))
    return out, g


def bwd_drop_brute(q, k, v, dout, bits, rate, causal, scale=1.0, o_used=None):
    """Gradients (dq, dk, dv) of the masked forward, the mask held fixed."""
    q, k, v, dout = _f64(q), _f64(k), _f64(v), _f64(dout)
    B, H, N, D = _shape4(q)
    b = _bits(bits, B, H, N, D)
    ou = None if o_used is None else _f64(o_used)
    dq, dk, dv = np.empty_like(q), np.empty_like(q), np.empty_like(q)
    _load().fmo_bwd_drop_brute(_ptr(q), _ptr(k), _ptr(v), _ptr(dout), _ptr(ou), _uptr(b),
                               B, H, N, D, int(causal), float(scale), float(rate),
                               _ptr(dq), _ptr(dk), _ptr(dv))
    return dq, dk, dv

"""ctypes binding of the Fastmax C ABI (include/fastmax.h).

Argument marshalling only: every step of the computation runs in the HIP
library.  Tensors are PyTorch device tensors (they supply memory and the
stream); the library must be built (``python -m paper_2402_07901_amd.build``)
and fails loudly when it is missing.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
# the sanitizer tier (tests/test_sanitize.py) points FASTMAX_LIB at the build
# whose host code carries AddressSanitizer/UBSan
LIB_PATH = os.environ.get("FASTMAX_LIB", os.path.join(_HERE, "libfastmax.so"))

F32 = 0
BF16 = 1

OK = 0
EINVAL = -1
EUNSUPPORTED = -2
ENULL = -3
EALIGN = -4
EWORKSPACE = -5
EHIP = -6

_lib = None


class FastmaxError(RuntimeError):
    def __init__(self, code: int, what: str):
        super().__init__(f"{what}: {strerror(code)} (code {code})")
        self.code = code


def lib():
    """The loaded libfastmax.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} not found: build it with `python -m paper_2402_07901_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        vp, i, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
        L.fastmax_workspace_bytes.argtypes = [i, i, i, i, i, i, i, i]
        L.fastmax_workspace_bytes.restype = sz
        L.fastmax_fwd.argtypes = [vp, vp, vp, vp, vp, i, i, i, i, i, i, i, vp, sz, vp]
        L.fastmax_fwd.restype = i
        L.fastmax_bwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, i, i, i, i, i, i, i,
                                  vp, sz, vp]
        L.fastmax_bwd.restype = i
        f = ctypes.c_float
        L.fastmax_fwd_scaled.argtypes = [vp, vp, vp, vp, vp, i, i, i, i, i, i, f, i, vp, sz, vp]
        L.fastmax_fwd_scaled.restype = i
        L.fastmax_bwd_scaled.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, i, i, i, i, i, i, f,
                                         i, vp, sz, vp]
        L.fastmax_bwd_scaled.restype = i
        u64 = ctypes.c_uint64
        L.fastmax_dropout_mask_words.argtypes = [i]
        L.fastmax_dropout_mask_words.restype = sz
        L.fastmax_dropout_mask.argtypes = [vp, i, i, i, i, f, u64, vp]
        L.fastmax_dropout_mask.restype = i
        L.fastmax_dropout_workspace_bytes.argtypes = [i, i, i, i, i, i, i]
        L.fastmax_dropout_workspace_bytes.restype = sz
        L.fastmax_fwd_dropout.argtypes = [vp, vp, vp, vp, vp, vp, f, i, i, i, i, i, f, i, vp, sz,
                                          vp]
        L.fastmax_fwd_dropout.restype = i
        L.fastmax_bwd_dropout.argtypes = [vp, vp, vp, vp, vp, vp, vp, f, vp, vp, vp, i, i, i, i,
                                          i, f, i, vp, sz, vp]
        L.fastmax_bwd_dropout.restype = i
        L.fastmax_fwd_noalloc.argtypes = [vp, vp, vp, vp, vp, i, i, i, i, i, i, f, i, vp]
        L.fastmax_fwd_noalloc.restype = i
        L.fastmax_set_scan_segments.argtypes = [i]
        L.fastmax_set_scan_segments.restype = i
        L.fastmax_strerror.argtypes = [i]
        L.fastmax_strerror.restype = ctypes.c_char_p
        L.fastmax_version.restype = ctypes.c_char_p
        _lib = L
    return _lib


def strerror(code: int) -> str:
    return lib().fastmax_strerror(int(code)).decode()


def version() -> str:
    return lib().fastmax_version().decode()


# fastmax_set_scan_segments modes
SCAN_SEGMENTS_AUTO, SCAN_SEGMENTS_OFF, SCAN_SEGMENTS_ON, SCAN_SEGMENTS_REBUILD = 0, 1, 2, 3


def set_scan_segments(mode: int) -> int:
    """Process-wide segment mode of the causal MFMA scans; returns the previous one."""
    return lib().fastmax_set_scan_segments(int(mode))


def workspace_bytes(B, H, N, D, p, causal, dt, backward=False) -> int:
    return int(lib().fastmax_workspace_bytes(B, H, N, D, p, int(causal), dt, int(backward)))


def _ptr(t):
    if t is None:
        return None
    return ctypes.c_void_p(t.data_ptr()) if hasattr(t, "data_ptr") else ctypes.c_void_p(t)


def _stream(stream):
    """The stream argument as a handle: ``stream`` as given (a torch stream or
    a raw handle), else the current device's current stream."""
    if stream is None:
        import torch
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else stream)


def _stream_of(stream, device):
    """``stream``, or the current stream of ``device`` when None."""
    if stream is None:
        import torch
        return torch.cuda.current_stream(device)
    return stream


def _on(device):
    """Context that makes ``device`` current for a library call (the library
    runs its kernels, and requires its stream to be, on the current device)."""
    import torch
    return torch.cuda.device(device)


def _dtype_code(t):
    import torch
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def fastmax_fwd_raw(q, k, v, out, g, B, H, N, D, p, causal, dt, workspace, ws_bytes, stream,
                    scale=None):
    """Direct call of fastmax_fwd (fastmax_fwd_scaled when ``scale`` is given)
    with raw pointers/ints; returns the code."""
    if scale is None:
        return lib().fastmax_fwd(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(g), B, H, N, D, p,
                                 int(causal), dt, _ptr(workspace), ws_bytes, _stream(stream))
    return lib().fastmax_fwd_scaled(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(g), B, H, N, D,
                                    p, int(causal), float(scale), dt, _ptr(workspace), ws_bytes,
                                    _stream(stream))


def fastmax_bwd_raw(q, k, v, out, dout, g, dq, dk, dv, B, H, N, D, p, causal, dt, workspace,
                    ws_bytes, stream, scale=None):
    if scale is None:
        return lib().fastmax_bwd(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(dout), _ptr(g),
                                 _ptr(dq), _ptr(dk), _ptr(dv), B, H, N, D, p, int(causal), dt,
                                 _ptr(workspace), ws_bytes, _stream(stream))
    return lib().fastmax_bwd_scaled(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(dout), _ptr(g),
                                    _ptr(dq), _ptr(dk), _ptr(dv), B, H, N, D, p, int(causal),
                                    float(scale), dt, _ptr(workspace), ws_bytes,
                                    _stream(stream))


# the library's per-GPU scratch size for fastmax_fwd_noalloc (include/fastmax.h)
NOALLOC_MAX_WORKSPACE_BYTES = 64 << 20


def fastmax_fwd_noalloc_raw(q, k, v, out, g, B, H, N, D, p, causal, dt, stream, scale=1.0):
    """Direct call of fastmax_fwd_noalloc with raw pointers/ints; returns the code."""
    return lib().fastmax_fwd_noalloc(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(g), B, H, N, D,
                                     p, int(causal), float(scale), dt, _stream(stream))


def fastmax_fwd_noalloc(q, k, v, out, g=None, p=2, causal=False, stream=None, scale=None):
    """fastmax_fwd into caller-provided ``out`` (and ``g``) with the library's
    per-GPU scratch as workspace: nothing is allocated."""
    B, H, N, D = _check_args(q, k=(k, "like_q"), v=(v, "like_q"), out=(out, "like_q"),
                             g=(g, "g"))
    with _on(q.device):
        rc = fastmax_fwd_noalloc_raw(q, k, v, out, g, B, H, N, D, p, causal, _dtype_code(q),
                                     _stream_of(stream, q.device), 1.0 if scale is None else scale)
    if rc != OK:
        raise FastmaxError(rc, "fastmax_fwd_noalloc")
    return out, g


def _check_args(q, **tensors):
    """Shape, dtype, layout and device checks the C ABI cannot make (it sees
    pointers only): q is a contiguous [B, H, N, D] tensor on a GPU; every
    other tensor is contiguous, on q's device, with the shape and dtype
    its entry names ("like_q": q's; "g": float32 [B, H, N]; "bits": int32
    [B, H, N, words]; "workspace": any dtype).  Returns (B, H, N, D)."""
    import torch
    if q.dim() != 4:
        raise ValueError(f"q must be [B, H, N, D], got shape {tuple(q.shape)}")
    B, H, N, D = q.shape
    if not q.is_contiguous():
        raise ValueError("q must be contiguous")
    want = {"like_q": (tuple(q.shape), q.dtype), "g": ((B, H, N), torch.float32)}
    for name, (t, kind) in tensors.items():
        if t is None:
            continue
        if kind == "bits":
            shape, dtype = (B, H, N, mask_words(D)), torch.int32
        elif kind == "workspace":
            shape, dtype = tuple(t.shape), t.dtype
        else:
            shape, dtype = want[kind]
        if tuple(t.shape) != shape:
            raise ValueError(f"{name} must have shape {shape}, got {tuple(t.shape)}")
        if t.dtype != dtype:
            raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
        if t.device != q.device:
            raise ValueError(f"{name} is on {t.device}, q on {q.device}")
    if q.device.type != "cuda":
        raise ValueError(f"the tensors must be on a GPU, q is on {q.device}")
    return B, H, N, D


def _alloc_ws(nbytes, device):
    import torch
    if nbytes == 0:
        return None
    return torch.empty(nbytes, dtype=torch.uint8, device=device)


def fastmax_fwd(q, k, v, p=2, causal=False, out=None, g=None, want_g=True, workspace=None,
                stream=None, scale=None):
    """O = Fastmax(q, k, v) for [B, H, N, D] device tensors; returns (O, G).
    ``scale``: score scale (weights f_p(scale * q^.k^)); None = the definition."""
    import torch
    B, H, N, D = _check_args(q, k=(k, "like_q"), v=(v, "like_q"), out=(out, "like_q"),
                             g=(g, "g"), workspace=(workspace, "workspace"))
    dt = _dtype_code(q)
    if out is None:
        out = torch.empty_like(q)
    if g is None and want_g:
        g = torch.empty((B, H, N), dtype=torch.float32, device=q.device)
    need = workspace_bytes(B, H, N, D, p, causal, dt, False)
    if workspace is None:
        workspace = _alloc_ws(need, q.device)
    ws_n = 0 if workspace is None else workspace.numel() * workspace.element_size()
    with _on(q.device):
        rc = fastmax_fwd_raw(q, k, v, out, g, B, H, N, D, p, causal, dt, workspace, ws_n,
                             _stream_of(stream, q.device), scale)
    if rc != OK:
        raise FastmaxError(rc, "fastmax_fwd")
    return out, g


def fastmax_bwd(q, k, v, out, dout, g, p=2, causal=False, dq=None, dk=None, dv=None,
                workspace=None, stream=None, scale=None):
    """Gradients (dq, dk, dv) of sum(dout * O); ``scale`` as in the forward."""
    import torch
    B, H, N, D = _check_args(q, k=(k, "like_q"), v=(v, "like_q"), out=(out, "like_q"),
                             dout=(dout, "like_q"), g=(g, "g"), dq=(dq, "like_q"),
                             dk=(dk, "like_q"), dv=(dv, "like_q"),
                             workspace=(workspace, "workspace"))
    dt = _dtype_code(q)
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(q) if dk is None else dk
    dv = torch.empty_like(q) if dv is None else dv
    need = workspace_bytes(B, H, N, D, p, causal, dt, True)
    if workspace is None:
        workspace = _alloc_ws(need, q.device)
    ws_n = 0 if workspace is None else workspace.numel() * workspace.element_size()
    with _on(q.device):
        rc = fastmax_bwd_raw(q, k, v, out, dout, g, dq, dk, dv, B, H, N, D, p, causal, dt,
                             workspace, ws_n, _stream_of(stream, q.device), scale)
    if rc != OK:
        raise FastmaxError(rc, "fastmax_bwd")
    return dq, dk, dv


# ---------------------------------------------------------------------------
# Quadratic-term dropout (Sec. 2.4, dropout paragraph; Fig. 2), p = 2.  Keep
# bits are an int32 tensor [B, H, N, mask_words(D)] holding the uint32 words.
# ---------------------------------------------------------------------------
def mask_words(D) -> int:
    """uint32 words per token of a keep-bit row (0 for an unsupported D)."""
    return int(lib().fastmax_dropout_mask_words(int(D)))


def fastmax_dropout_mask_raw(bits, B, H, N, D, rate, seed, stream):
    return lib().fastmax_dropout_mask(_ptr(bits), B, H, N, D, float(rate),
                                      ctypes.c_uint64(int(seed)), _stream(stream))


def dropout_mask(B, H, N, D, rate, seed, device="cuda", stream=None):
    """Philox4x32-10 keep bits for the quadratic features of every key token."""
    import torch
    bits = torch.empty((B, H, N, mask_words(D)), dtype=torch.int32, device=device)
    with _on(bits.device):
        rc = fastmax_dropout_mask_raw(bits, B, H, N, D, rate, seed,
                                      _stream_of(stream, bits.device))
    if rc != OK:
        raise FastmaxError(rc, "fastmax_dropout_mask")
    return bits


def dropout_workspace_bytes(B, H, N, D, causal, dt, backward=False) -> int:
    return int(lib().fastmax_dropout_workspace_bytes(B, H, N, D, int(causal), dt,
                                                     int(bool(backward))))


def fastmax_fwd_dropout_raw(q, k, v, out, g, bits, rate, B, H, N, D, causal, scale, dt,
                            workspace, ws_bytes, stream):
    return lib().fastmax_fwd_dropout(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(g), _ptr(bits),
                                     float(rate), B, H, N, D, int(causal), float(scale), dt,
                                     _ptr(workspace), ws_bytes, _stream(stream))


def fastmax_bwd_dropout_raw(q, k, v, out, dout, g, bits, rate, dq, dk, dv, B, H, N, D, causal,
                            scale, dt, workspace, ws_bytes, stream):
    return lib().fastmax_bwd_dropout(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(dout), _ptr(g),
                                     _ptr(bits), float(rate), _ptr(dq), _ptr(dk), _ptr(dv), B, H,
                                     N, D, int(causal), float(scale), dt, _ptr(workspace),
                                     ws_bytes, _stream(stream))


def fastmax_fwd_dropout(q, k, v, bits, rate, causal=False, scale=None, out=None, g=None,
                        workspace=None, stream=None):
    """Forward with the quadratic features of the keys masked by ``bits``
    (kept ones scaled by 1/(1 - rate)); returns (O, G)."""
    import torch
    B, H, N, D = _check_args(q, k=(k, "like_q"), v=(v, "like_q"), bits=(bits, "bits"),
                             out=(out, "like_q"), g=(g, "g"),
                             workspace=(workspace, "workspace"))
    dt = _dtype_code(q)
    out = torch.empty_like(q) if out is None else out
    if g is None:
        g = torch.empty((B, H, N), dtype=torch.float32, device=q.device)
    if workspace is None:
        workspace = _alloc_ws(dropout_workspace_bytes(B, H, N, D, causal, dt, False), q.device)
    ws_n = 0 if workspace is None else workspace.numel() * workspace.element_size()
    with _on(q.device):
        rc = fastmax_fwd_dropout_raw(q, k, v, out, g, bits, rate, B, H, N, D, causal,
                                     1.0 if scale is None else scale, dt, workspace, ws_n,
                                     _stream_of(stream, q.device))
    if rc != OK:
        raise FastmaxError(rc, "fastmax_fwd_dropout")
    return out, g


def fastmax_bwd_dropout(q, k, v, out, dout, g, bits, rate, causal=False, scale=None, dq=None,
                        dk=None, dv=None, workspace=None, stream=None):
    """Gradients (dq, dk, dv) of sum(dout * O) for the forward with the same bits."""
    import torch
    B, H, N, D = _check_args(q, k=(k, "like_q"), v=(v, "like_q"), out=(out, "like_q"),
                             dout=(dout, "like_q"), g=(g, "g"), bits=(bits, "bits"),
                             dq=(dq, "like_q"), dk=(dk, "like_q"), dv=(dv, "like_q"),
                             workspace=(workspace, "workspace"))
    dt = _dtype_code(q)
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(q) if dk is None else dk
    dv = torch.empty_like(q) if dv is None else dv
    if workspace is None:
        workspace = _alloc_ws(dropout_workspace_bytes(B, H, N, D, causal, dt, True), q.device)
    ws_n = 0 if workspace is None else workspace.numel() * workspace.element_size()
    with _on(q.device):
        rc = fastmax_bwd_dropout_raw(q, k, v, out, dout, g, bits, rate, dq, dk, dv, B, H, N, D,
                                     causal, 1.0 if scale is None else scale, dt, workspace,
                                     ws_n, _stream_of(stream, q.device))
    if rc != OK:
        raise FastmaxError(rc, "fastmax_bwd_dropout")
    return dq, dk, dv

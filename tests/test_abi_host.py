"""Host-only tests of the C ABI (no GPU needed).

Every call here carries at least one invalid argument, so the library must
reject it during host validation, before any HIP call; the fake device
pointers are never dereferenced.
"""
import ctypes
import os
import re

import pytest

from paper_2402_07901_amd import fastmax as fm

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fastmax.h")

pytestmark = pytest.mark.skipif(not os.path.exists(fm.LIB_PATH),
                                reason="libfastmax.so not built")

A = 0x100000  # 16-byte aligned fake pointer (never dereferenced)


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(fastmax_[a-z_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert {"fastmax_fwd", "fastmax_bwd", "fastmax_workspace_bytes",
            "fastmax_strerror", "fastmax_version"} <= set(names)
    L = ctypes.CDLL(fm.LIB_PATH)
    for n in names:
        assert hasattr(L, n), n


def test_strerror_and_version():
    for code in (fm.OK, fm.EINVAL, fm.EUNSUPPORTED, fm.ENULL, fm.EALIGN, fm.EWORKSPACE,
                 fm.EHIP, 12345):
        s = fm.strerror(code)
        assert isinstance(s, str) and s
    assert re.match(r"^\d+\.\d+\.\d+$", fm.version())


def fwd(q=A, k=A, v=A, out=A, g=None, B=1, H=1, N=8, D=64, p=2, causal=1, dt=fm.BF16,
        ws=None, wsb=0):
    return fm.lib().fastmax_fwd(ctypes.c_void_p(q), ctypes.c_void_p(k), ctypes.c_void_p(v),
                                ctypes.c_void_p(out), ctypes.c_void_p(g) if g else None, B, H,
                                N, D, p, causal, dt, ctypes.c_void_p(ws) if ws else None, wsb,
                                None)


def bwd(ptrs=None, B=1, H=1, N=8, D=64, p=2, causal=1, dt=fm.BF16, ws=None, wsb=0):
    ptrs = ptrs or [A] * 9
    cp = [ctypes.c_void_p(x) if x else None for x in ptrs]
    return fm.lib().fastmax_bwd(*cp, B, H, N, D, p, causal, dt,
                                ctypes.c_void_p(ws) if ws else None, wsb, None)


@pytest.mark.parametrize("kw,code", [
    (dict(B=0), fm.EINVAL), (dict(H=0), fm.EINVAL), (dict(N=0), fm.EINVAL),
    (dict(N=-5), fm.EINVAL), (dict(p=0), fm.EINVAL), (dict(p=3), fm.EINVAL),
    (dict(causal=2), fm.EINVAL), (dict(dt=7), fm.EINVAL),
    (dict(D=48), fm.EUNSUPPORTED), (dict(D=256), fm.EUNSUPPORTED), (dict(D=8), fm.EUNSUPPORTED),
    (dict(B=1 << 20, H=1 << 20, N=1 << 20), fm.EINVAL),
    (dict(B=(1 << 10) + 1, H=1 << 10), fm.EINVAL), (dict(N=(1 << 30) + 1), fm.EINVAL),
])
def test_fwd_rejects_bad_shape_args(kw, code):
    # also give a NULL q so that nothing could ever launch
    assert fwd(q=0, **kw) in (code, fm.ENULL)
    assert fwd(q=0, **kw) == code


def test_size_limits_are_inclusive():
    """2^20 heads and 2^30 tokens per head pass the size checks (a NULL q
    then stops the call before anything is enqueued); one more does not."""
    for B, H, N, D in ((1 << 10, 1 << 10, 1, 64), (1, 1, 1 << 30, 16)):
        assert fwd(q=0, B=B, H=H, N=N, D=D) == fm.ENULL
        assert bwd([0] + [A] * 8, B=B, H=H, N=N, D=D) == fm.ENULL
        assert fm.workspace_bytes(B, H, N, D, 2, 1, fm.BF16, False) > 0
    assert fm.workspace_bytes(1 << 10, (1 << 10) + 1, 1, 64, 2, 1, fm.BF16, False) == 0
    assert fm.workspace_bytes(1, 1, (1 << 30) + 1, 16, 2, 1, fm.BF16, False) == 0


@pytest.mark.parametrize("which", ["q", "k", "v", "out"])
def test_fwd_null(which):
    assert fwd(**{which: 0}) == fm.ENULL


@pytest.mark.parametrize("which", ["q", "k", "v", "out", "g"])
def test_fwd_misaligned(which):
    kw = {which: A + 4}
    kw.setdefault("q", A)
    assert fwd(**kw) == fm.EALIGN


def test_bwd_null_and_align():
    for i in range(9):
        ptrs = [A] * 9
        ptrs[i] = 0
        assert bwd(ptrs) == fm.ENULL
        ptrs = [A] * 9
        ptrs[i] = A + 8
        assert bwd(ptrs) == fm.EALIGN


def test_bwd_workspace_checks():
    need = fm.workspace_bytes(1, 1, 8, 64, 2, True, fm.BF16, True)
    assert need > 0
    assert bwd(ws=None, wsb=0) == fm.EWORKSPACE
    assert bwd(ws=A, wsb=need - 1) == fm.EWORKSPACE
    ptrs = [A] * 9
    assert bwd(ptrs, ws=A + 4, wsb=need, p=5) == fm.EINVAL


def test_fwd_workspace_checks():
    # the segmented non-causal path (bf16, D = 64, p = 2) needs a workspace
    need = fm.workspace_bytes(1, 2, 1000, 64, 2, False, fm.BF16, False)
    assert need > 0
    assert fwd(causal=0, N=1000, H=2, ws=None, wsb=0) == fm.EWORKSPACE
    assert fwd(causal=0, N=1000, H=2, ws=A, wsb=need - 1) == fm.EWORKSPACE
    assert fwd(causal=0, N=1000, H=2, ws=A + 4, wsb=need) == fm.EALIGN
    # sized for the whole problem: grows with the number of heads and tokens
    assert fm.workspace_bytes(1, 8, 131072, 64, 2, False, fm.BF16, False) > need
    # the causal MFMA scan keeps q^ and k^ in fp16: 256 bytes per row
    need_c = fm.workspace_bytes(1, 2, 1000, 64, 2, True, fm.BF16, False)
    assert need_c >= 2 * 1000 * 256
    assert fwd(causal=1, N=1000, H=2, ws=None, wsb=0) == fm.EWORKSPACE
    assert fwd(causal=1, N=1000, H=2, ws=A, wsb=need_c - 1) == fm.EWORKSPACE
    # the float32 kernels (generic and MFMA) need segment sums only when few heads must be
    # spread over the CUs; with many heads (>= 256 workgroups) none
    for D, p, causal, dt in ((64, 2, False, fm.F32), (32, 2, False, fm.BF16),
                             (32, 1, True, fm.F32), (16, 2, True, fm.F32)):
        assert fm.workspace_bytes(1, 2, 1000, D, p, causal, dt, False) > 0
        assert fm.workspace_bytes(64, 8, 1000, D, p, causal, dt, False) == 0
    # fewer keys than one 128-token chunk: the generic kernel (segment states)
    assert fm.workspace_bytes(1, 2, 127, 64, 2, False, fm.BF16, False) > 0
    assert fm.workspace_bytes(1, 2, 128, 64, 2, False, fm.BF16, False) > 0
    # a single 16-token chunk cannot be split
    assert fm.workspace_bytes(1, 1, 16, 32, 2, True, fm.F32, False) == 0


def test_bwd_rejects_bad_args():
    assert bwd(B=0) == fm.EINVAL
    assert bwd(D=100) == fm.EUNSUPPORTED
    assert bwd(p=3) == fm.EINVAL


def test_workspace_bytes():
    for D in (16, 32, 64, 128):
        for p in (1, 2):
            for causal in (0, 1):
                for dt in (fm.F32, fm.BF16):
                    nf = fm.workspace_bytes(2, 3, 100, D, p, causal, dt, False)
                    nb = fm.workspace_bytes(2, 3, 100, D, p, causal, dt, True)
                    # fp32 dq^ and dk^ plus two floats per row, on every path
                    assert nf >= 0 and nb >= 4 * 2 * 3 * 100 * (2 * D + 2)
    assert fm.workspace_bytes(0, 1, 1, 64, 2, 1, fm.BF16, True) == 0
    assert fm.workspace_bytes(1, 1, 1, 65, 2, 1, fm.BF16, True) == 0


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(fm, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(fm, "_lib", None)
    with pytest.raises(RuntimeError, match="not found"):
        fm.lib()


def fwd_scaled(scale, q=A, B=1, H=1, N=8, D=64, p=2, causal=1, dt=fm.BF16):
    return fm.lib().fastmax_fwd_scaled(ctypes.c_void_p(q) if q else None, ctypes.c_void_p(A),
                                       ctypes.c_void_p(A), ctypes.c_void_p(A), None, B, H, N, D,
                                       p, causal, ctypes.c_float(scale), dt, None, 0, None)


def bwd_scaled(scale, first=A, B=1, H=1, N=8, D=64, p=2, causal=1, dt=fm.BF16):
    cp = [ctypes.c_void_p(first) if first else None] + [ctypes.c_void_p(A)] * 8
    return fm.lib().fastmax_bwd_scaled(*cp, B, H, N, D, p, causal, ctypes.c_float(scale), dt,
                                       None, 0, None)


@pytest.mark.parametrize("scale", [0.0, -0.5, 1.5, float("nan"), float("inf"), -float("inf")])
def test_scaled_entry_points_reject_bad_scale(scale):
    # every other argument is valid: the scale check alone must stop the call
    # (fake pointers, nothing may launch)
    assert fwd_scaled(scale) == fm.EINVAL
    assert bwd_scaled(scale) == fm.EINVAL


def test_scaled_entry_points_validate_the_rest():
    for s in (1.0, 1.0 / 64, 0.125):
        assert fwd_scaled(s, q=0) == fm.ENULL
        assert bwd_scaled(s, first=0) == fm.ENULL
        assert fwd_scaled(s, D=48) == fm.EUNSUPPORTED
        assert bwd_scaled(s, p=3) == fm.EINVAL
        assert fwd_scaled(s, q=A + 4) == fm.EALIGN
    # causal bf16 D = 64 p = 2 needs a workspace (none given)
    assert fwd_scaled(0.5) == fm.EWORKSPACE
    assert bwd_scaled(0.5) == fm.EWORKSPACE


# --------------------------------------------------------------------------
# Quadratic-term dropout entry points
# --------------------------------------------------------------------------
def test_dropout_mask_words():
    for D, nw in ((16, 5), (32, 17), (64, 65), (128, 258), (8, 0), (256, 0)):
        assert fm.lib().fastmax_dropout_mask_words(D) == nw, D


def test_dropout_workspace():
    """Backward: the generic float32 backward's (c, dq^, dk^ and dv in fp32,
    plus segment states when few heads are split into segments); causal
    forward: the non-causal one (256-byte aligned, the generic kernels' p = 2
    segment states) plus the masked in-chunk weights, 16 x 16 floats per
    chunk of 16 tokens."""
    L = fm.lib()
    for B, H, N, D in ((1, 1, 700, 16), (4, 16, 8192, 64), (1, 8, 4096, 128), (2, 3, 33, 32)):
        for causal in (0, 1):
            a = L.fastmax_dropout_workspace_bytes(B, H, N, D, causal, fm.BF16, 1)
            base = 4 * B * H * N * (1 + 3 * D)
            assert a >= base, (B, H, N, D)
            if (B, H) == (4, 16):   # 832 (head, slice) items: no segments
                assert a == base
        a_nc = L.fastmax_dropout_workspace_bytes(B, H, N, D, 0, fm.BF16, 0)
        a_c = L.fastmax_dropout_workspace_bytes(B, H, N, D, 1, fm.BF16, 0)
        assert a_c == (a_nc + 255) // 256 * 256 + B * H * ((N + 15) // 16) * 16 * 16 * 4, (B, H, N, D)


def mask_call(bits=A, B=1, H=1, N=8, D=64, rate=0.1, seed=1):
    return fm.lib().fastmax_dropout_mask(ctypes.c_void_p(bits) if bits else None, B, H, N, D,
                                         ctypes.c_float(rate), ctypes.c_uint64(seed), None)


def test_dropout_mask_rejects():
    assert mask_call(rate=-0.1) == fm.EINVAL
    assert mask_call(rate=1.0) == fm.EINVAL
    assert mask_call(rate=float("nan")) == fm.EINVAL
    assert mask_call(bits=None) == fm.ENULL
    assert mask_call(bits=A + 2) == fm.EALIGN
    assert mask_call(D=48) == fm.EUNSUPPORTED
    assert mask_call(N=0) == fm.EINVAL


def fwd_drop(ptrs=None, rate=0.1, B=1, H=1, N=8, D=64, causal=1, scale=1.0, dt=fm.BF16,
             ws=None, wsb=0):
    ptrs = ptrs or [A] * 6     # q, k, v, out, g, bits
    cp = [ctypes.c_void_p(x) if x else None for x in ptrs]
    return fm.lib().fastmax_fwd_dropout(*cp, ctypes.c_float(rate), B, H, N, D, causal,
                                        ctypes.c_float(scale), dt,
                                        ctypes.c_void_p(ws) if ws else None, wsb, None)


def bwd_drop(ptrs=None, rate=0.1, B=1, H=1, N=8, D=64, causal=1, scale=1.0, dt=fm.BF16,
             ws=None, wsb=0):
    ptrs = ptrs or [A] * 10    # q, k, v, out, dout, g, bits, dq, dk, dv
    cp = [ctypes.c_void_p(x) if x else None for x in ptrs]
    return fm.lib().fastmax_bwd_dropout(*cp[:7], ctypes.c_float(rate), *cp[7:], B, H, N, D,
                                        causal, ctypes.c_float(scale), dt,
                                        ctypes.c_void_p(ws) if ws else None, wsb, None)


def test_fwd_dropout_rejects():
    for rate in (-1e-3, 1.0, float("nan")):
        assert fwd_drop(rate=rate) == fm.EINVAL
    assert fwd_drop(scale=0.0) == fm.EINVAL
    assert fwd_drop(D=24) == fm.EUNSUPPORTED
    assert fwd_drop(causal=2) == fm.EINVAL
    assert fwd_drop(ptrs=[A, A, A, A, A, None]) == fm.ENULL
    assert fwd_drop(ptrs=[A, A, A, A, A, A + 2]) == fm.EALIGN
    assert fwd_drop(ptrs=[A, A, A + 8, A, A, A]) == fm.EALIGN
    # few heads and many tokens: segment states, so a workspace is required
    assert fwd_drop(N=100000, causal=0) == fm.EWORKSPACE
    # causal: the masked in-chunk weights always need one
    assert fwd_drop(N=8, causal=1) == fm.EWORKSPACE


def test_bwd_dropout_rejects():
    assert bwd_drop(rate=1.5) == fm.EINVAL
    for i in range(10):
        ptrs = [A] * 10
        ptrs[i] = None
        assert bwd_drop(ptrs=ptrs) == fm.ENULL, i
    ptrs = [A] * 10
    ptrs[6] = A + 1
    assert bwd_drop(ptrs=ptrs) == fm.EALIGN
    assert bwd_drop() == fm.EWORKSPACE   # the backward always needs one
    need = fm.lib().fastmax_dropout_workspace_bytes(1, 1, 8, 64, 1, fm.BF16, 1)
    assert bwd_drop(ws=A, wsb=need - 1) == fm.EWORKSPACE


def fwd_noalloc(q=A, k=A, v=A, out=A, g=None, B=1, H=1, N=8, D=64, p=2, causal=1, dt=fm.BF16,
                scale=1.0):
    return fm.lib().fastmax_fwd_noalloc(ctypes.c_void_p(q), ctypes.c_void_p(k),
                                        ctypes.c_void_p(v), ctypes.c_void_p(out),
                                        ctypes.c_void_p(g) if g else None, B, H, N, D, p, causal,
                                        float(scale), dt, None)


@pytest.mark.parametrize("kw,code", [
    (dict(B=0), fm.EINVAL), (dict(p=3), fm.EINVAL), (dict(dt=7), fm.EINVAL),
    (dict(scale=0.0), fm.EINVAL), (dict(scale=1.5), fm.EINVAL), (dict(D=48), fm.EUNSUPPORTED),
    (dict(q=0), fm.ENULL), (dict(out=0), fm.ENULL), (dict(k=A + 8), fm.EALIGN),
    (dict(g=A + 4), fm.EALIGN),
])
def test_fwd_noalloc_validates_like_the_forward(kw, code):
    assert fwd_noalloc(**kw) == code


def test_fwd_noalloc_rejects_problems_beyond_its_scratch():
    """A problem whose forward workspace exceeds the 64 MiB scratch is
    rejected on the host (EWORKSPACE), one that fits is not rejected for
    its size (with a NULL q it then fails on the pointer check)."""
    lim = fm.NOALLOC_MAX_WORKSPACE_BYTES
    big = dict(B=1, H=1, N=1 << 20, D=64, p=2, causal=1, dt=fm.BF16)
    need = fm.workspace_bytes(big["B"], big["H"], big["N"], big["D"], big["p"], big["causal"],
                              big["dt"])
    assert need > lim
    assert fwd_noalloc(**big) == fm.EWORKSPACE
    small = dict(B=1, H=1, N=4096, D=64, p=2, causal=1, dt=fm.BF16)
    assert 0 < fm.workspace_bytes(1, 1, 4096, 64, 2, 1, fm.BF16) <= lim
    assert fwd_noalloc(q=0, **small) == fm.ENULL
    # the largest causal bf16 D = 64 problems the header quotes fit exactly
    assert fm.workspace_bytes(1, 1, 260594, 64, 2, 1, fm.BF16) <= lim
    assert fm.workspace_bytes(1, 1, 260595, 64, 2, 1, fm.BF16) > lim
    assert fm.workspace_bytes(1, 46, 4096, 64, 2, 1, fm.BF16) <= lim
    assert fm.workspace_bytes(1, 47, 4096, 64, 2, 1, fm.BF16) > lim
    # and the D = 128 p = 2 ones (four partial numerators per token)
    assert fm.workspace_bytes(1, 8, 4064, 128, 2, 1, fm.BF16) <= lim
    assert fm.workspace_bytes(1, 8, 4065, 128, 2, 1, fm.BF16) > lim
    assert fm.workspace_bytes(1, 1, 11081, 128, 2, 1, fm.BF16) <= lim
    assert fm.workspace_bytes(1, 1, 11082, 128, 2, 1, fm.BF16) > lim


def test_scan_segment_mode_setter():
    """fastmax_set_scan_segments: unknown modes are rejected, valid ones
    return the previous mode; the workspace sizes do not depend on it."""
    L = fm.lib()
    for bad in (-1, 4, 1 << 30):
        assert L.fastmax_set_scan_segments(bad) == fm.EINVAL
    prev = fm.set_scan_segments(fm.SCAN_SEGMENTS_AUTO)
    try:
        sizes = []
        for mode in (fm.SCAN_SEGMENTS_OFF, fm.SCAN_SEGMENTS_ON, fm.SCAN_SEGMENTS_REBUILD,
                     fm.SCAN_SEGMENTS_AUTO):
            before = fm.set_scan_segments(mode)
            assert fm.set_scan_segments(mode) == mode
            sizes.append([fm.workspace_bytes(8, 12, 4096, 64, 2, 1, fm.BF16, bw) for bw in (0, 1)])
            assert before in (0, 1, 2, 3)
        assert all(x == sizes[0] for x in sizes)
    finally:
        fm.set_scan_segments(prev)


# ---------------------------------------------------------------------------
# The binding's tensor checks (the C ABI sees pointers only, so a tensor of
# the wrong shape, dtype, layout or device must be refused before any call).
# CPU tensors: every case below fails a check before the library is reached.
# ---------------------------------------------------------------------------
def _qkv(shape=(1, 2, 8, 16), dtype=None):
    import torch
    dtype = dtype or torch.float32
    return [torch.zeros(shape, dtype=dtype) for _ in range(3)]


def test_binding_rejects_mismatched_tensors():
    import torch
    q, k, v = _qkv()
    with pytest.raises(ValueError, match=r"q must be \[B, H, N, D\]"):
        fm.fastmax_fwd(q[0], k[0], v[0])
    with pytest.raises(ValueError, match="k must have shape"):
        fm.fastmax_fwd(q, k[:, :, :4], v)
    with pytest.raises(ValueError, match="v must be torch.float32"):
        fm.fastmax_fwd(q, k, v.to(torch.bfloat16))
    with pytest.raises(ValueError, match="v must be contiguous"):
        fm.fastmax_fwd(q, k, v.transpose(2, 3).contiguous().transpose(2, 3))
    with pytest.raises(ValueError, match="q must be contiguous"):
        fm.fastmax_fwd(q.transpose(2, 3).contiguous().transpose(2, 3), k, v)
    with pytest.raises(ValueError, match="g must have shape"):
        fm.fastmax_fwd(q, k, v, g=torch.zeros(1, 2, 7))
    with pytest.raises(ValueError, match="g must be torch.float32"):
        fm.fastmax_fwd(q, k, v, g=torch.zeros(1, 2, 8, dtype=torch.float64))
    with pytest.raises(ValueError, match="dout must have shape"):
        fm.fastmax_bwd(q, k, v, q, k[:, :1], torch.zeros(1, 2, 8))
    with pytest.raises(ValueError, match="dq must be torch.float32"):
        fm.fastmax_bwd(q, k, v, q, k, torch.zeros(1, 2, 8), dq=q.to(torch.bfloat16))
    with pytest.raises(ValueError, match="bits must have shape"):
        fm.fastmax_fwd_dropout(q, k, v, torch.zeros(1, 2, 8, 1, dtype=torch.int32), 0.1)
    with pytest.raises(ValueError, match="bits must be torch.int32"):
        fm.fastmax_fwd_dropout(q, k, v, torch.zeros(1, 2, 8, fm.mask_words(16)), 0.1)
    with pytest.raises(ValueError, match="workspace must be contiguous"):
        fm.fastmax_fwd(q, k, v, workspace=torch.zeros(8, 8, dtype=torch.uint8).t())


def test_binding_refuses_host_tensors():
    """Consistent tensors on the CPU: refused as not on a GPU (a kernel given
    host pointers would fault), by every wrapper."""
    import torch
    q, k, v = _qkv()
    g = torch.zeros(1, 2, 8)
    bits = torch.zeros(1, 2, 8, fm.mask_words(16), dtype=torch.int32)
    calls = [lambda: fm.fastmax_fwd(q, k, v),
             lambda: fm.fastmax_bwd(q, k, v, q, q, g),
             lambda: fm.fastmax_fwd_noalloc(q, k, v, q.clone(), g),
             lambda: fm.fastmax_fwd_dropout(q, k, v, bits, 0.1),
             lambda: fm.fastmax_bwd_dropout(q, k, v, q, q, g, bits, 0.1)]
    for call in calls:
        with pytest.raises(ValueError, match="must be on a GPU"):
            call()


@pytest.mark.parametrize("B,H,N,D,backward", [
    (1, 1 << 18, 1, 128, False),   # float32 MFMA forward: 2^23 workgroups of 512 threads
    (1, 1 << 18, 1, 128, True),
    (1 << 10, 1 << 10, 1, 64, True),   # bf16 D = 64 backward: 2^23 moment-gradient workgroups
])
def test_grids_beyond_the_dispatch_limits_are_unsupported(B, H, N, D, backward):
    """Within the size limits but with a launch grid of 2^32 work-items: the
    launcher refuses it before its first launch (no HIP call is made, so this
    runs without a GPU) and the call returns FASTMAX_EUNSUPPORTED."""
    need = fm.workspace_bytes(B, H, N, D, 2, 1, fm.BF16, backward)
    assert need > 0
    if backward:
        rc = bwd(B=B, H=H, N=N, D=D, ws=A, wsb=need)
    else:
        rc = fwd(B=B, H=H, N=N, D=D, ws=A, wsb=need)
    assert rc == fm.EUNSUPPORTED

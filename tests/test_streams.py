"""GPU test: every entry point accepts a stream of the current device other
than the null one (the library asks HIP for the stream's device and refuses
another device's), and its results there equal those on the default stream:
the forward and backward on the fp16 MFMA path (bit for bit: deterministic)
and on the float32 kernels (within their run-to-run rounding), the keep bits
(bit for bit), the masked forward, and the allocation-free forward.
"""
import numpy as np
import pytest

from paper_2402_07901_amd import fastmax as fm
from paper_2402_07901_amd.inputs import make_inputs

from gpu_util import max_rel, say, to_dev, to_f64

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fm.lib()
    yield
    torch.cuda.synchronize()


def same(a, b, exact, label):
    import torch
    if exact:
        assert torch.equal(a.view(torch.int16) if a.dtype == torch.bfloat16 else a,
                           b.view(torch.int16) if b.dtype == torch.bfloat16 else b), label
    else:
        e = max_rel(to_f64(a), to_f64(b))
        assert e <= 2e-5, (label, e)


@pytest.mark.parametrize("D,dtype,causal", [(64, "bf16", True), (64, "bf16", False),
                                            (32, "f32", True)])
def test_side_stream_matches_default_stream(D, dtype, causal):
    import torch
    label = f"side stream D={D} {dtype} causal={causal}"
    say(label)
    inp = make_inputs(1, 2, 700, D, 5100 + D, dtype, with_dout=True)
    q, k, v, do = (to_dev(inp[n], dtype) for n in ("q", "k", "v", "dout"))
    o0, g0 = fm.fastmax_fwd(q, k, v, p=2, causal=causal)
    d0 = fm.fastmax_bwd(q, k, v, o0, do, g0, p=2, causal=causal)
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    assert s.cuda_stream != 0
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        o1, g1 = fm.fastmax_fwd(q, k, v, p=2, causal=causal, stream=s)
        d1 = fm.fastmax_bwd(q, k, v, o1, do, g1, p=2, causal=causal, stream=s)
        out = torch.empty_like(q)
        g2 = torch.empty_like(g0)
        fm.fastmax_fwd_noalloc(q, k, v, out, g2, p=2, causal=causal, stream=s)
    s.synchronize()
    exact = dtype == "bf16"
    for nm, a, b in (("O", o0, o1), ("G", g0, g1), ("O noalloc", o0, out), ("G noalloc", g0, g2)):
        same(a, b, exact, (label, nm))
    for nm, a, b in zip(("dq", "dk", "dv"), d0, d1):
        same(a, b, exact, (label, nm))


def test_side_stream_dropout():
    import torch
    say("side stream dropout")
    B, H, N, D = 1, 2, 300, 32
    inp = make_inputs(B, H, N, D, 5200, "f32")
    q, k, v = (to_dev(inp[n], "f32") for n in ("q", "k", "v"))
    b0 = fm.dropout_mask(B, H, N, D, 0.2, 77)
    o0, g0 = fm.fastmax_fwd_dropout(q, k, v, b0, 0.2, causal=True)
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        b1 = fm.dropout_mask(B, H, N, D, 0.2, 77, stream=s)
        o1, g1 = fm.fastmax_fwd_dropout(q, k, v, b1, 0.2, causal=True, stream=s)
    s.synchronize()
    assert torch.equal(b0, b1)
    same(o0, o1, False, "dropout O")
    same(g0, g1, False, "dropout G")

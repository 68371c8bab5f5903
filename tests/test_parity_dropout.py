"""GPU parity of the quadratic-term dropout (Sec. 2.4, dropout paragraph;
Fig. 2) against the fp64 oracle.

* fastmax_dropout_mask: the Philox4x32-10 keep bits, bit for bit against the
  oracle's generator (itself pinned to the published known-answer vectors).
* fastmax_fwd_dropout / fastmax_bwd_dropout: O, G and the gradients for keep
  bits drawn by the ORACLE (never by the GPU), against the oracle's explicit
  masked weights, every D, causal and not, float32 and bf16 I/O, single and
  multiple chunks, ragged tails, the segmented scans (few heads), score
  scales, and rate 0 with every bit kept (the plain p = 2 call).
"""
import numpy as np
import pytest

import oracle
from paper_2402_07901_amd import fastmax as fm
from paper_2402_07901_amd.inputs import make_inputs

from gpu_util import TOL, max_rel, say, to_dev, to_f64

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fm.lib()
    yield
    torch.cuda.synchronize()


def bits_dev(bits):
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int32)).cuda()


def f32(r):
    """The rate as the float32 the ABI receives (the oracle uses the same value)."""
    return float(np.float32(r))


@pytest.mark.parametrize("shape", [(2, 3, 50, 16), (1, 2, 37, 32), (1, 2, 33, 64),
                                   (1, 1, 5, 128)])
@pytest.mark.parametrize("rate", [0.0, 0.1, 0.5, 0.999])
def test_mask_bit_exact(shape, rate):
    import torch
    B, H, N, D = shape
    seed = 0x9E3779B97F4A7C15 ^ (N * 1000 + D)
    say(f"mask {shape} rate={rate}")
    got = fm.dropout_mask(B, H, N, D, rate, seed)
    torch.cuda.synchronize()
    want = oracle.dropout_mask(B, H, N, D, f32(rate), seed)
    np.testing.assert_array_equal(got.cpu().numpy().view(np.uint32), want)


def test_mask_large():
    """2.6 M words over 8 heads of 5000 tokens, every word checked."""
    import torch
    B, H, N, D = 2, 4, 5000, 64
    got = fm.dropout_mask(B, H, N, D, 0.25, 12345)
    torch.cuda.synchronize()
    want = oracle.dropout_mask(B, H, N, D, 0.25, 12345)
    np.testing.assert_array_equal(got.cpu().numpy().view(np.uint32), want)


def fwd_case(B, H, N, D, causal, dtype, rate, seed, scale=1.0, label=""):
    import torch
    inp = make_inputs(B, H, N, D, seed, dtype)
    bits = oracle.dropout_mask(B, H, N, D, f32(rate), seed * 7919 + 1)
    q, k, v = (to_dev(inp[n], dtype) for n in ("q", "k", "v"))
    o, g = fm.fastmax_fwd_dropout(q, k, v, bits_dev(bits), rate, causal=causal, scale=scale)
    torch.cuda.synchronize()
    ref_o, ref_g = oracle.fwd_drop_brute(inp["q64"], inp["k64"], inp["v64"], bits, f32(rate),
                                         causal, scale=scale)
    out = to_f64(o)
    gg = g.cpu().numpy().astype(np.float64)
    assert np.isfinite(out).all()
    e = max_rel(out, ref_o)
    eg = float((np.abs(gg - ref_g) / np.abs(ref_g)).max())
    say(f"{label}: E_O={e:.3e} E_G={eg:.3e}")
    assert e <= TOL[dtype], (label, e)
    assert eg <= TOL[dtype], (label, eg)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("D", [16, 32, 64])
@pytest.mark.parametrize("N", [1, 17, 100])
def test_fwd_dropout(N, D, causal, dtype):
    label = f"fwd dropout N={N} D={D} causal={causal} {dtype}"
    say(label)
    fwd_case(2, 2, N, D, causal, dtype, 0.3, 1000 + N + D, label=label)


@pytest.mark.parametrize("causal", [False, True])
def test_fwd_dropout_d128(causal):
    label = f"fwd dropout D=128 causal={causal}"
    say(label)
    fwd_case(1, 2, 40, 128, causal, "f32", 0.2, 1100, label=label)


@pytest.mark.parametrize("rate", [0.05, 0.9])
@pytest.mark.parametrize("scale", [1.0, 0.125])
def test_fwd_dropout_rates_and_scale(rate, scale):
    label = f"fwd dropout rate={rate} scale={scale}"
    say(label)
    fwd_case(1, 3, 70, 64, True, "f32", rate, 1200, scale=scale, label=label)


@pytest.mark.parametrize("causal", [False, True])
def test_fwd_dropout_segments(causal):
    """One head of 700 tokens: the moment states of segments of chunks are
    built in parallel (with the masked key features), then prefix-summed."""
    label = f"fwd dropout segments causal={causal}"
    say(label)
    fwd_case(1, 1, 700, 16, causal, "f32", 0.4, 1300, label=label)


def bwd_case(B, H, N, D, causal, dtype, rate, seed, scale=1.0, label="", floor=None):
    """floor: a lower bound for the error's denominator (the tensor's max |ref|),
    for gradients that are exactly zero."""
    import torch
    inp = make_inputs(B, H, N, D, seed, dtype, with_dout=True)
    bits = oracle.dropout_mask(B, H, N, D, f32(rate), seed * 31 + 5)
    q, k, v = (to_dev(inp[n], dtype) for n in ("q", "k", "v"))
    do = to_dev(inp["dout"], dtype)
    bd = bits_dev(bits)
    o, g = fm.fastmax_fwd_dropout(q, k, v, bd, rate, causal=causal, scale=scale)
    dq, dk, dv = fm.fastmax_bwd_dropout(q, k, v, o, do, g, bd, rate, causal=causal, scale=scale)
    torch.cuda.synchronize()
    rq, rk, rv = oracle.bwd_drop_brute(inp["q64"], inp["k64"], inp["v64"], inp["dout64"], bits,
                                       f32(rate), causal, scale=scale)
    for nm, got, ref in (("dq", dq, rq), ("dk", dk, rk), ("dv", dv, rv)):
        x = to_f64(got)
        if floor is None:
            e = max_rel(x, ref)
        else:
            e = float(np.abs(x - ref).max() / max(np.abs(ref).max(), floor))
        say(f"{label} {nm}: E={e:.3e}")
        assert np.isfinite(x).all()
        assert e <= TOL[dtype], (label, nm, e)
    return inp


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("D", [16, 32, 64])
def test_bwd_dropout(D, causal, dtype):
    label = f"bwd dropout D={D} causal={causal} {dtype}"
    say(label)
    bwd_case(1, 2, 37, D, causal, dtype, 0.3, 1400 + D, label=label)


@pytest.mark.parametrize("causal", [False, True])
def test_bwd_dropout_d128_and_scale(causal):
    label = f"bwd dropout D=128 causal={causal} scale=1/sqrt(128)"
    say(label)
    bwd_case(1, 1, 21, 128, causal, "f32", 0.2, 1500, scale=float(np.float32(128 ** -0.5)),
             label=label)


@pytest.mark.parametrize("causal", [False, True])
def test_bwd_dropout_segments(causal):
    """One head of 700 tokens: both backward scans run in segments."""
    label = f"bwd dropout segments causal={causal}"
    say(label)
    bwd_case(1, 1, 700, 16, causal, "f32", 0.4, 1600, label=label)


@pytest.mark.parametrize("causal", [False, True])
def test_rate0_all_kept_is_the_plain_call(causal):
    """Every bit kept at rate 0 gives f_2: the dropout kernels agree with the
    plain p = 2 call (same float32 kernels, up to their run-to-run rounding)."""
    import torch
    B, H, N, D = 1, 2, 150, 32
    inp = make_inputs(B, H, N, D, 1700, "f32", with_dout=True)
    q, k, v = (to_dev(inp[n], "f32") for n in ("q", "k", "v"))
    do = to_dev(inp["dout"], "f32")
    bits = bits_dev(oracle.dropout_mask(B, H, N, D, 0.0, 3))
    o0, g0 = fm.fastmax_fwd(q, k, v, p=2, causal=causal)
    o1, g1 = fm.fastmax_fwd_dropout(q, k, v, bits, 0.0, causal=causal)
    d0 = fm.fastmax_bwd(q, k, v, o0, do, g0, p=2, causal=causal)
    d1 = fm.fastmax_bwd_dropout(q, k, v, o0, do, g0, bits, 0.0, causal=causal)
    torch.cuda.synchronize()
    for nm, a, b in (("O", o0, o1), ("G", g0, g1)) + tuple(zip(("dq", "dk", "dv"), d0, d1)):
        e = max_rel(to_f64(b), to_f64(a))
        say(f"rate 0 causal={causal} {nm}: E={e:.3e}")
        assert e <= 2e-5, (nm, e)


def test_workload_dropout_fwdbwd_bf16():
    """The bench's dropout workload (B8 H12 N4096 D64, causal, bf16, rate 0.1):
    two whole heads of the forward against the oracle's factorised masked
    forward; the backward on a 256-token problem of the same recipe (the
    brute-force gradient is quadratic in N)."""
    import torch
    from paper_2402_07901_amd.inputs import WORKLOADS, workload_inputs
    w = WORKLOADS["fwdbwd_causal_bf16"]
    rate = 0.1
    say(f"{w.name} dropout")
    inp = workload_inputs(w)
    bits = oracle.dropout_mask(w.B, w.H, w.N, w.D, f32(rate), 2024)
    q, k, v = (to_dev(inp[n], w.dtype) for n in ("q", "k", "v"))
    o, g = fm.fastmax_fwd_dropout(q, k, v, bits_dev(bits), rate, causal=True)
    torch.cuda.synchronize()
    out = to_f64(o)
    for b, h in ((0, 0), (w.B - 1, w.H - 1)):
        sl = (slice(b, b + 1), slice(h, h + 1))
        ro, rg = oracle.fwd_drop_fact(inp["q64"][sl], inp["k64"][sl], inp["v64"][sl], bits[sl],
                                      f32(rate), True)
        e = max_rel(out[sl], ro)
        eg = float((np.abs(g.cpu().numpy()[sl] - rg) / np.abs(rg)).max())
        say(f"{w.name} dropout head ({b},{h}): E_O={e:.3e} E_G={eg:.3e}")
        assert e <= TOL[w.dtype] and eg <= TOL[w.dtype], (b, h, e, eg)
    bwd_case(2, 2, 256, 64, True, "bf16", rate, 1800, label="dropout bwd N=256 D=64 bf16")


def test_padding_bits_are_ignored():
    """Bits past D(D+1)/2 in a token's last word carry nothing: setting them
    all leaves O, G and the gradients unchanged (D = 16: 136 features, 5 words,
    the last 24 bits padding)."""
    import torch
    B, H, N, D, rate = 1, 2, 40, 16, 0.3
    inp = make_inputs(B, H, N, D, 1900, "f32", with_dout=True)
    bits = oracle.dropout_mask(B, H, N, D, f32(rate), 77)
    padded = bits.copy()
    padded[..., -1] |= np.uint32(0xFFFFFFFF) << np.uint32(136 % 32)
    assert not np.array_equal(bits, padded)
    q, k, v = (to_dev(inp[n], "f32") for n in ("q", "k", "v"))
    do = to_dev(inp["dout"], "f32")
    outs = []
    for b in (bits, padded):
        bd = bits_dev(b)
        o, g = fm.fastmax_fwd_dropout(q, k, v, bd, rate, causal=True)
        grads = fm.fastmax_bwd_dropout(q, k, v, o, do, g, bd, rate, causal=True)
        torch.cuda.synchronize()
        outs.append([to_f64(t) for t in (o, g) + tuple(grads)])
    for a, b in zip(*outs):
        assert max_rel(b, a) <= 2e-6


@pytest.mark.parametrize("causal", [False, True])
def test_generator_feeds_the_masked_calls(causal):
    """End to end: bits drawn on the GPU by fastmax_dropout_mask drive the
    masked forward; the oracle draws its own bits from the same seed."""
    import torch
    B, H, N, D, rate, seed = 2, 2, 90, 32, 0.25, 0xDEADBEEFCAFE
    inp = make_inputs(B, H, N, D, 2000, "bf16")
    q, k, v = (to_dev(inp[n], "bf16") for n in ("q", "k", "v"))
    bd = fm.dropout_mask(B, H, N, D, rate, seed)
    o, g = fm.fastmax_fwd_dropout(q, k, v, bd, rate, causal=causal)
    torch.cuda.synchronize()
    bits = oracle.dropout_mask(B, H, N, D, f32(rate), seed)
    ref_o, ref_g = oracle.fwd_drop_fact(inp["q64"], inp["k64"], inp["v64"], bits, f32(rate),
                                        causal)
    e = max_rel(to_f64(o), ref_o)
    eg = float((np.abs(g.cpu().numpy() - ref_g) / np.abs(ref_g)).max())
    say(f"generator -> fwd causal={causal}: E_O={e:.3e} E_G={eg:.3e}")
    assert e <= TOL["bf16"] and eg <= TOL["bf16"], (e, eg)


def test_fwd_dropout_past_65535_chunks():
    """One head of 1,048,616 tokens (65539 chunks of 16, more than the 65535
    blocks of a grid's y dimension): the masked in-chunk weights are computed
    by blocks that stride over the chunks; every row of the tail against the
    oracle's factorised masked forward."""
    import torch
    B, H, N, D, rate = 1, 1, 65536 * 16 + 40, 16, 0.2
    inp = make_inputs(B, H, N, D, 2100, "f32")
    bits = oracle.dropout_mask(B, H, N, D, f32(rate), 5)
    q, k, v = (to_dev(inp[n], "f32") for n in ("q", "k", "v"))
    o, g = fm.fastmax_fwd_dropout(q, k, v, bits_dev(bits), rate, causal=True)
    torch.cuda.synchronize()
    ref_o, ref_g = oracle.fwd_drop_fact(inp["q64"], inp["k64"], inp["v64"], bits, f32(rate), True)
    tail = slice(65535 * 16 - 20, N)
    e = max_rel(to_f64(o)[0, 0, tail], ref_o[0, 0, tail])
    eg = float((np.abs(g.cpu().numpy()[0, 0, tail] - ref_g[0, 0, tail]) / np.abs(ref_g[0, 0, tail])).max())
    say(f"N={N}: tail E_O={e:.3e} E_G={eg:.3e}")
    assert e <= TOL["f32"] and eg <= TOL["f32"], (e, eg)


def test_workload_rate0_matches_the_mfma_path():
    """At the bench's full shape (B8 H12 N4096 D64, causal, bf16): every bit
    kept at rate 0 makes the masked calls compute f_2, so the float32 dropout
    kernels must agree with the plain calls, which take the (independently
    oracle-checked) MFMA forward and backward here -- forward and backward
    compared on every element."""
    import torch
    from paper_2402_07901_amd.inputs import WORKLOADS, workload_inputs
    w = WORKLOADS["fwdbwd_causal_bf16"]
    inp = workload_inputs(w, want64=False)
    q, k, v = (to_dev(inp[n], w.dtype) for n in ("q", "k", "v"))
    do = to_dev(inp["dout"], w.dtype)
    bits = fm.dropout_mask(w.B, w.H, w.N, w.D, 0.0, 1)
    o0, g0 = fm.fastmax_fwd(q, k, v, p=2, causal=True)
    o1, g1 = fm.fastmax_fwd_dropout(q, k, v, bits, 0.0, causal=True)
    d0 = fm.fastmax_bwd(q, k, v, o0, do, g0, p=2, causal=True)
    d1 = fm.fastmax_bwd_dropout(q, k, v, o0, do, g0, bits, 0.0, causal=True)
    torch.cuda.synchronize()
    for nm, a, b in (("O", o0, o1), ("G", g0, g1)) + tuple(zip(("dq", "dk", "dv"), d0, d1)):
        e = max_rel(to_f64(b), to_f64(a))
        say(f"{w.name} rate 0 vs MFMA {nm}: E={e:.3e}")
        assert e <= TOL["bf16"], (nm, e)


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("N", [1, 16, 17])
def test_bwd_dropout_edges(N, causal):
    """One token, exactly one chunk, and one chunk plus one token.  With one
    token O = v whatever q and k are, so the exact dq and dk are zero: errors
    are measured against the gradient scale max|dO| max|v| where the exact
    gradient is smaller."""
    label = f"bwd dropout edge N={N} causal={causal}"
    say(label)
    inp = make_inputs(1, 2, N, 64, 2200 + N, "f32", with_dout=True)
    floor = float(np.abs(inp["dout64"]).max() * np.abs(inp["v64"]).max())
    bwd_case(1, 2, N, 64, causal, "f32", 0.5, 2200 + N, label=label, floor=floor)

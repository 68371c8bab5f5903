"""GPU parity cases aimed at the MFMA paths (D = 64, p = 2, bf16 I/O).

The non-causal path splits the sequence into segments whose fp32 partial
moments are summed and converted to fp16 with power-of-two scales; the causal
path scans 128-token chunks.  These cases span several segments, token blocks
and chunks with ragged tails, extreme value magnitudes (the scales), the
long-sequence recipe at N = 8192, run-to-run determinism, and the row
normalisation property (rows of A sum to 1, Eq. "valid": constant V gives
O = V) at the full workload sizes.
"""
import numpy as np
import pytest

import oracle
from paper_2402_07901_amd import fastmax as fm
from paper_2402_07901_amd.inputs import (WORKLOADS, bf16_bits_to_f64, f32_to_bf16_bits,
                                         make_inputs, workload_inputs)

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


def fwd(inp, causal):
    import torch
    q, k, v = (to_dev(inp[n], "bf16") for n in ("q", "k", "v"))
    o, g = fm.fastmax_fwd(q, k, v, p=2, causal=causal)
    torch.cuda.synchronize()
    return o, g


def compare_brute(inp, o, g, causal, label):
    ref_o, ref_g = oracle.fwd_brute(inp["q64"], inp["k64"], inp["v64"], 2, causal)
    out = to_f64(o)
    gg = g.cpu().numpy().astype(np.float64)
    assert np.isfinite(out).all(), label
    e = max_rel(out, ref_o)
    eg = float((np.abs(gg - ref_g) / np.abs(ref_g)).max())
    say(f"{label}: E_O={e:.3e} E_G={eg:.3e}")
    assert e <= TOL["bf16"], (label, e)
    assert eg <= TOL["bf16"], (label, eg)


def with_v_scaled(inp, e):
    """Same inputs with v multiplied by 2^e (exact in bf16 while in range)."""
    v32 = (inp["v64"] * 2.0 ** e).astype(np.float32)
    bits = f32_to_bf16_bits(v32)
    out = dict(inp)
    out["v"] = bits
    out["v64"] = bf16_bits_to_f64(bits)
    assert np.array_equal(out["v64"], inp["v64"] * 2.0 ** e)
    return out


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("shape", [(1, 3, 128), (2, 1, 129), (1, 2, 1000), (2, 3, 777),
                                   (1, 1, 4097)])
def test_multi_segment_vs_brute(shape, causal):
    B, H, N = shape
    label = f"mfma B={B} H={H} N={N} causal={causal}"
    say(label)
    inp = make_inputs(B, H, N, 64, 500 + N, "bf16")
    o, g = fwd(inp, causal)
    compare_brute(inp, o, g, causal, label)


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("e", [-60, -20, 20, 60])
def test_value_scale_extremes(e, causal):
    label = f"mfma v*2^{e} causal={causal}"
    say(label)
    inp = with_v_scaled(make_inputs(1, 2, 700, 64, 900, "bf16"), e)
    o, g = fwd(inp, causal)
    compare_brute(inp, o, g, causal, label)


def test_long_recipe_at_8192_sampled():
    """The long non-causal recipe (5% of tokens scaled by 4) at N = 8192."""
    w = WORKLOADS["long_noncausal_bf16"]
    N = 8192
    say(f"{w.name} at N={N}")
    inp = make_inputs(w.B, w.H, N, w.D, w.key, "bf16", w.mask_frac, w.mask_scale)
    o, g = fwd(inp, False)
    rng = np.random.default_rng(7)
    rows = np.unique(np.concatenate([np.arange(0, w.B * w.H * N, N), np.arange(N - 1, w.B * w.H * N, N),
                                     rng.integers(0, w.B * w.H * N, 40)])).astype(np.int64)
    ref_o, ref_g = oracle.fwd_rows(inp["q64"], inp["k64"], inp["v64"], 2, False, rows)
    out = to_f64(o).reshape(-1, w.D)[rows]
    gg = g.cpu().numpy().astype(np.float64).reshape(-1)[rows]
    e = max_rel(out, ref_o)
    eg = float((np.abs(gg - ref_g) / ref_g).max())
    say(f"sampled rows={rows.size} E_O={e:.3e} E_G={eg:.3e}")
    assert e <= TOL["bf16"] and eg <= TOL["bf16"]


@pytest.mark.parametrize("causal", [False, True])
def test_deterministic(causal):
    import torch
    inp = make_inputs(2, 2, 3000, 64, 77, "bf16")
    q, k, v = (to_dev(inp[n], "bf16") for n in ("q", "k", "v"))
    o1, g1 = fm.fastmax_fwd(q, k, v, p=2, causal=causal)
    o2, g2 = fm.fastmax_fwd(q, k, v, p=2, causal=causal)
    torch.cuda.synchronize()
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    assert torch.equal(g1, g2)


@pytest.mark.parametrize("name", ["long_noncausal_bf16", "gpt_causal_bf16"])
def test_constant_v_full_size(name):
    """Rows of the normalised score matrix sum to 1, so a V whose rows are
    all equal comes back unchanged, at the full workload size (every row)."""
    import torch
    w = WORKLOADS[name]
    say(f"constant V at {w.name}")
    gen = torch.Generator(device="cuda").manual_seed(11)
    shape = (w.B, w.H, w.N, w.D)
    q = torch.randn(shape, device="cuda", generator=gen).to(torch.bfloat16)
    k = torch.randn(shape, device="cuda", generator=gen).to(torch.bfloat16)
    row = (torch.arange(w.D, device="cuda", dtype=torch.float32) - 20.0) * 0.37
    row = row.to(torch.bfloat16)
    v = row.expand(shape).contiguous()
    o, g = fm.fastmax_fwd(q, k, v, p=2, causal=w.causal)
    torch.cuda.synchronize()
    err = ((o.float() - row.float()).abs().max() / row.float().abs().max()).item()
    say(f"max|O - v| / max|v| = {err:.3e}")
    assert err <= 1e-2
    # p = 2: G_i >= (number of keys) / 2
    nk = (torch.arange(1, w.N + 1, device="cuda", dtype=torch.float32) if w.causal
          else torch.full((w.N,), float(w.N), device="cuda"))
    assert bool((g >= nk / 2 * (1 - 1e-5)).all())


@pytest.mark.parametrize("shape", [(1, 1, 129), (1, 2, 300), (2, 1, 777)])
def test_bwd_multi_chunk_vs_brute(shape):
    """Causal backward across several 128-token chunks (the moment scans in
    both directions) with ragged tails, against the fp64 explicit backward."""
    from test_parity_gpu import bwd_case
    B, H, N = shape
    label = f"mfma bwd B={B} H={H} N={N}"
    say(label)
    inp = make_inputs(B, H, N, 64, 700 + N, "bf16", with_dout=True)
    bwd_case(inp, 2, True, "bf16", label=label)


@pytest.mark.parametrize("ev,ed", [(-40, 0), (40, 0), (0, -40), (0, 40)])
def test_bwd_value_scale_extremes(ev, ed):
    """v and dO scaled by powers of two (exact in bf16): the gradients scale
    accordingly and the per-head fp16 scales must follow."""
    from test_parity_gpu import bwd_case
    label = f"mfma bwd v*2^{ev} dO*2^{ed}"
    say(label)
    inp = make_inputs(1, 1, 400, 64, 800, "bf16", with_dout=True)
    inp = with_v_scaled(inp, ev)
    d32 = (inp["dout64"] * 2.0 ** ed).astype(np.float32)
    inp["dout"] = f32_to_bf16_bits(d32)
    inp["dout64"] = bf16_bits_to_f64(inp["dout"])
    bwd_case(inp, 2, True, "bf16", label=label)


def test_bwd_single_token():
    """N = 1: O_1 = v_1 whatever q and k are, so dq = dk = 0 exactly and
    dv = dO.  The computed dq, dk are pure rounding of u~ . v' = u.v - c
    (exactly 0); they are bounded by the size of the terms that cancel,
    eps (1 + |s|) sum_j |u_j v_j| max|k^| / std(q) with eps = 2e-2."""
    import torch
    inp = make_inputs(1, 3, 1, 64, 901, "bf16", with_dout=True)
    q, k, v, do = (to_dev(inp[n], "bf16") for n in ("q", "k", "v", "dout"))
    o, g = fm.fastmax_fwd(q, k, v, p=2, causal=True)
    dq, dk, dv = fm.fastmax_bwd(q, k, v, o, do, g, p=2, causal=True)
    torch.cuda.synchronize()
    e = max_rel(to_f64(dv), inp["dout64"])
    say(f"N=1: E(dv vs dO)={e:.3e}")
    assert e <= TOL["bf16"]
    for hh in range(3):
        qq, kk_, vv, dd = (inp[n][0, hh, 0] for n in ("q64", "k64", "v64", "dout64"))
        qh = (qq - qq.mean()) / qq.std()
        kh = (kk_ - kk_.mean()) / kk_.std()
        s = float(qh @ kh)
        G = 1.0 + s + s * s / 2.0
        mag = (1.0 + abs(s)) * float(np.abs(dd / G * vv).sum())
        bq = 2e-2 * mag * np.abs(kh).max() / qq.std()
        bk = 2e-2 * mag * np.abs(qh).max() / kk_.std()
        aq = float(np.abs(to_f64(dq)[0, hh, 0]).max())
        ak = float(np.abs(to_f64(dk)[0, hh, 0]).max())
        say(f"N=1 head {hh}: |dq|={aq:.3e} (bound {bq:.3e}) |dk|={ak:.3e} (bound {bk:.3e})")
        assert aq <= bq and ak <= bk


def test_bwd_long_ragged_vs_brute():
    """Backward over 33 chunks with a ragged tail (N = 4173): every chunk of
    the forward and reverse moment scans, against the fp64 explicit backward."""
    from test_parity_gpu import bwd_case
    label = "mfma bwd B=1 H=1 N=4173"
    say(label)
    inp = make_inputs(1, 1, 4173, 64, 4173, "bf16", with_dout=True)
    bwd_case(inp, 2, True, "bf16", label=label)


def test_bwd_deterministic():
    """The backward has one writer per output element (no atomics): two calls
    give bit-identical gradients."""
    import torch
    inp = make_inputs(2, 3, 1500, 64, 31, "bf16", with_dout=True)
    q, k, v, do = (to_dev(inp[n], "bf16") for n in ("q", "k", "v", "dout"))
    o, g = fm.fastmax_fwd(q, k, v, p=2, causal=True)
    r1 = fm.fastmax_bwd(q, k, v, o, do, g, p=2, causal=True)
    r2 = fm.fastmax_bwd(q, k, v, o, do, g, p=2, causal=True)
    torch.cuda.synchronize()
    for a, b in zip(r1, r2):
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))


def test_user_stream_ordering():
    """Forward and backward enqueued on a caller's non-default stream: results
    equal the default-stream ones, and work the caller enqueues after the call
    on its stream sees the finished outputs."""
    import torch
    inp = make_inputs(1, 4, 2000, 64, 47, "bf16", with_dout=True)
    q, k, v, do = (to_dev(inp[n], "bf16") for n in ("q", "k", "v", "dout"))
    o0, g0 = fm.fastmax_fwd(q, k, v, p=2, causal=True)
    ref = fm.fastmax_bwd(q, k, v, o0, do, g0, p=2, causal=True)
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        o1, g1 = fm.fastmax_fwd(q, k, v, p=2, causal=True, stream=s)
        got = fm.fastmax_bwd(q, k, v, o1, do, g1, p=2, causal=True, stream=s)
        # consumers on the same stream, before any host synchronisation
        sums = [x.float().sum() for x in got]
    s.synchronize()
    assert torch.equal(o0.view(torch.int16), o1.view(torch.int16))
    for a, b, sm in zip(ref, got, sums):
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))
        assert float(sm) == float(b.float().sum())


@pytest.mark.parametrize("shape", [(1, 1, 128), (1, 2, 129), (2, 1, 700), (1, 1, 4097)])
def test_bwd_noncausal_mfma_vs_brute(shape):
    """Non-causal backward on the MFMA kernels (N >= 128): dv by the
    non-causal forward kernels with queries and keys exchanged, dq^ and dk^
    by the moment-gradient scans against the totals; every entry against the
    fp64 explicit backward."""
    from test_parity_gpu import bwd_case
    B, H, N = shape
    label = f"mfma bwd non-causal B={B} H={H} N={N}"
    say(label)
    inp = make_inputs(B, H, N, 64, 1700 + N, "bf16", with_dout=True)
    bwd_case(inp, 2, False, "bf16", label=label)


@pytest.mark.parametrize("ev,ed", [(-40, 0), (40, 0), (0, -40), (0, 40)])
def test_bwd_noncausal_value_scale_extremes(ev, ed):
    from test_parity_gpu import bwd_case
    label = f"mfma bwd non-causal v*2^{ev} dO*2^{ed}"
    say(label)
    inp = make_inputs(1, 1, 400, 64, 1800, "bf16", with_dout=True)
    inp = with_v_scaled(inp, ev)
    d32 = (inp["dout64"] * 2.0 ** ed).astype(np.float32)
    inp["dout"] = f32_to_bf16_bits(d32)
    inp["dout64"] = bf16_bits_to_f64(inp["dout"])
    bwd_case(inp, 2, False, "bf16", label=label)


def test_bwd_noncausal_deterministic():
    import torch
    inp = make_inputs(2, 2, 1500, 64, 1900, "bf16", with_dout=True)
    q, k, v, do = (to_dev(inp[n], "bf16") for n in ("q", "k", "v", "dout"))
    o, g = fm.fastmax_fwd(q, k, v, p=2, causal=False)
    r1 = fm.fastmax_bwd(q, k, v, o, do, g, p=2, causal=False)
    r2 = fm.fastmax_bwd(q, k, v, o, do, g, p=2, causal=False)
    torch.cuda.synchronize()
    for a, b in zip(r1, r2):
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))

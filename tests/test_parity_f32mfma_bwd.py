"""GPU parity of the float32 MFMA backward (p = 2; D in {16, 32, 128} with
float32 or bf16 I/O, D = 64 with float32 I/O; causal and non-causal) against
the fp64 oracle's brute-force backward (the explicit N x N gradient of the
Sec. 2.2 definition, Sec. 2.5's formulas for the custom backward being an
identity for it).

dv comes from the forward's scan run over the reversed sequence; dq^ and dk^
from one gradient scan run forwards (keys' moments) and backwards (queries'
moments).  Shapes cover one token, ragged 32-token chunks, one and many
segments per head, four workgroups per (head, slice) at D = 128, and the
score scale.  Bars: float32 max|d - d_ref|/max|d_ref| <= 1e-4 per tensor and
head, bf16 I/O 2e-2.  A reference that is zero up to the oracle's rounding
(dq and dk of a one-token head, whose output v_1 does not depend on q or k)
is held to the same bar absolutely, relative to the gradient's natural size
max|dO| max|v| sqrt(D).
"""
import numpy as np
import pytest

import oracle
from paper_2402_07901_amd import fastmax as fm
from paper_2402_07901_amd.inputs import WORKLOADS, make_inputs, workload_inputs

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


def grad_err(x, ref, size):
    m = float(np.abs(ref).max())
    if m <= 1e-9 * size:
        return float(np.abs(x - ref).max()) / size
    return max_rel(x, ref)


def check(inp, causal, dtype, label, heads=None, scale=None):
    import torch
    q, k, v = (to_dev(inp[n], dtype) for n in ("q", "k", "v"))
    do = to_dev(inp["dout"], dtype)
    o, g = fm.fastmax_fwd(q, k, v, p=2, causal=causal, scale=scale)
    dq, dk, dv = fm.fastmax_bwd(q, k, v, o, do, g, p=2, causal=causal, scale=scale)
    torch.cuda.synchronize()
    tau = 1.0 if scale is None else scale
    B, H = inp["q64"].shape[:2]
    heads = heads or [(b, h) for b in range(B) for h in range(H)]
    worst = 0.0
    for b, h in heads:
        sl = (slice(b, b + 1), slice(h, h + 1))
        ref = oracle.bwd_brute(inp["q64"][sl], inp["k64"][sl], inp["v64"][sl],
                               inp["dout64"][sl], 2, causal, scale=tau)
        size = float(np.abs(inp["dout64"][sl]).max() * np.abs(inp["v64"][sl]).max())
        size *= np.sqrt(inp["q64"].shape[-1])
        for nm, got, r in zip(("dq", "dk", "dv"), (dq, dk, dv), ref):
            x = to_f64(got[sl])
            assert np.isfinite(x).all(), (label, nm, b, h)
            e = grad_err(x, r, size)
            worst = max(worst, e)
            assert e <= TOL[dtype], (label, nm, b, h, e)
    say(f"{label}: worst E={worst:.3e} over {len(heads)} heads")


CASES = [(D, causal, dtype) for D in (16, 32, 64, 128) for causal in (False, True)
         for dtype in ("f32", "bf16") if not (D == 64 and dtype == "bf16")]
SHAPES = [(1, 1, 1), (1, 2, 5), (2, 1, 31), (1, 1, 32), (1, 2, 33), (2, 3, 100), (1, 1, 257)]


@pytest.mark.parametrize("shape", SHAPES, ids=[f"B{b}H{h}N{n}" for b, h, n in SHAPES])
@pytest.mark.parametrize("case", CASES, ids=[f"D{d}-{'causal' if c else 'noncausal'}-{t}" for d, c, t in CASES])
def test_f32mfma_bwd_vs_brute(case, shape):
    D, causal, dtype = case
    B, H, N = shape
    inp = make_inputs(B, H, N, D, 9700 + D + N + 7 * H, dtype, with_dout=True)
    check(inp, causal, dtype, f"f32mfma bwd D={D} causal={causal} {dtype} B={B} H={H} N={N}")


@pytest.mark.parametrize("D", [16, 32, 64, 128])
@pytest.mark.parametrize("causal", [False, True])
def test_f32mfma_bwd_many_segments(D, causal):
    """One head of 2000 tokens: 63 chunks, up to 63 segments (8 at D = 128)
    whose moment sums are prefix-summed (causal, both directions) or
    totalled (non-causal)."""
    inp = make_inputs(1, 1, 2000, D, 9800 + D, "f32", with_dout=True)
    check(inp, causal, "f32", f"f32mfma bwd segments D={D} causal={causal}")


@pytest.mark.parametrize("tau", [1.0 / 32, 0.5])
@pytest.mark.parametrize("D", [32, 128])
def test_f32mfma_bwd_score_scale(D, tau):
    inp = make_inputs(1, 2, 300, D, 9900 + D, "f32", with_dout=True)
    check(inp, True, "f32", f"f32mfma bwd D={D} tau={tau}", scale=tau)


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("D,B,H,dtype", [(16, 16, 16, "f32"), (32, 8, 16, "bf16"),
                                         (128, 2, 4, "f32")])
def test_f32mfma_bwd_one_segment_per_head(D, B, H, dtype, causal):
    """Enough heads for one workgroup per (head, slice, part): no segment
    sums, the non-causal totals and outputs in one launch per scan."""
    inp = make_inputs(B, H, 100, D, 9950 + D, dtype, with_dout=True)
    heads = [(0, 0), (B - 1, H - 1), (B // 2, H // 3)]
    check(inp, causal, dtype, f"f32mfma bwd one segment D={D} {dtype} causal={causal}",
          heads=heads)


def test_f32mfma_bwd_lra_workload():
    """The LRA-shaped p = 2 workload (B2 H4 N2048 D32, causal, f32): two
    heads' full gradients against the brute-force oracle."""
    w = WORKLOADS["lra_causal_f32_p2"]
    inp = workload_inputs(w)
    if "dout" not in inp:
        rng = np.random.default_rng(123)
        d64 = rng.standard_normal(inp["q64"].shape)
        inp["dout"] = d64.astype(np.float32)
        inp["dout64"] = inp["dout"].astype(np.float64)
    check(inp, w.causal, w.dtype, w.name, heads=[(0, 0), (w.B - 1, w.H - 1)])


# ---------------------------------------------------------------------------
# p = 1 (f' = 1): every D and dtype, against the brute-force gradient with the
# per-entry first-order rounding bounds of gpu_util.grad_bounds (weights
# change sign and G_i may nearly cancel), through test_parity_gpu.bwd_case.
# ---------------------------------------------------------------------------
P1_BWD = [(D, causal, dtype) for D in (16, 32, 64, 128) for causal in (False, True)
          for dtype in ("f32", "bf16")]


@pytest.mark.parametrize("N", [1, 33, 100])
@pytest.mark.parametrize("case", P1_BWD, ids=[f"D{d}-{'causal' if c else 'noncausal'}-{t}" for d, c, t in P1_BWD])
def test_f32mfma_bwd_p1(case, N):
    from test_parity_gpu import bwd_case
    D, causal, dtype = case
    inp = make_inputs(1, 2, N, D, 9750 + D + N, dtype, with_dout=True)
    bwd_case(inp, 1, causal, dtype, label=f"f32mfma bwd p=1 D={D} causal={causal} {dtype} N={N}")


@pytest.mark.parametrize("causal", [False, True])
def test_f32mfma_bwd_p1_segments(causal):
    """One head of 2000 tokens (63 chunks, up to 63 segments), p = 1."""
    from test_parity_gpu import bwd_case
    inp = make_inputs(1, 1, 2000, 32, 9850, "f32", with_dout=True)
    bwd_case(inp, 1, causal, "f32", label=f"f32mfma bwd p=1 segments causal={causal}")

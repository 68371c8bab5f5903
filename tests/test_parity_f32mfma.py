"""GPU parity of the float32 MFMA forward (v_mfma_f32_16x16x4_f32; p = 2,
D in {16, 32, 128} with float32 or bf16 I/O, D = 64 with float32 I/O; causal
and non-causal) against the fp64 oracle: the explicit N x N definition
(Sec. 2.2, Eq. "tobeexpanded") on small shapes, the factorised oracle
(Sec. 2.4) on the full LRA-shaped and small configurations.

Shapes cover one token, ragged 32-token chunks, one and many segments per
head (few heads split a sequence into segments whose sums are prefix-summed),
and the score scale.  At D = 128 four workgroups share each (head, slice),
each holding a quarter of the feature tiles, and a finalize pass sums their
partial F and G; those cases run with one and with several segments.  Bars: float32 max|dO|/max|O_ref| <= 1e-4 and
max_i |dG_i|/G_i <= 1e-4; bf16 I/O 2e-2.
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


def check(inp, causal, dtype, label, ref="brute", scale=None):
    import torch
    q, k, v = (to_dev(inp[n], dtype) for n in ("q", "k", "v"))
    o, g = fm.fastmax_fwd(q, k, v, p=2, causal=causal, scale=scale)
    torch.cuda.synchronize()
    tau = 1.0 if scale is None else scale
    if ref == "brute":
        ro, rg = oracle.fwd_brute(inp["q64"], inp["k64"], inp["v64"], 2, causal, scale=tau)
    else:
        ro, rg = oracle.fwd_fact(inp["q64"], inp["k64"], inp["v64"], 2, causal)
    out = to_f64(o)
    gg = g.cpu().numpy().astype(np.float64)
    assert np.isfinite(out).all() and np.isfinite(gg).all(), label
    e = max_rel(out, ro)
    eg = float((np.abs(gg - rg) / np.abs(rg)).max())
    say(f"{label}: E_O={e:.3e} E_G={eg:.3e}")
    assert e <= TOL[dtype] and eg <= TOL[dtype], (label, e, eg)


CASES = [(D, causal, dtype) for D in (16, 32, 64, 128) for causal in (False, True)
         for dtype in ("f32", "bf16") if not (D == 64 and dtype == "bf16")]
SHAPES = [(1, 1, 1), (1, 2, 5), (2, 1, 31), (1, 1, 32), (1, 2, 33), (2, 3, 100), (1, 1, 257),
          (1, 1, 1000)]


@pytest.mark.parametrize("shape", SHAPES, ids=[f"B{b}H{h}N{n}" for b, h, n in SHAPES])
@pytest.mark.parametrize("case", CASES, ids=[f"D{d}-{'causal' if c else 'noncausal'}-{t}" for d, c, t in CASES])
def test_f32mfma_vs_brute(case, shape):
    D, causal, dtype = case
    B, H, N = shape
    inp = make_inputs(B, H, N, D, 9100 + D + N + 7 * H, dtype)
    check(inp, causal, dtype, f"f32mfma D={D} causal={causal} {dtype} B={B} H={H} N={N}")


@pytest.mark.parametrize("D", [16, 32, 64, 128])
@pytest.mark.parametrize("causal", [False, True])
def test_f32mfma_many_segments(D, causal):
    """One head, 4000 tokens: up to 125 segments of one 32-token chunk each
    (8 at D = 128, whose head spans 32 workgroups), their sums prefix-summed
    (causal) or totalled (non-causal)."""
    inp = make_inputs(1, 1, 4000, D, 9300 + D, "f32")
    check(inp, causal, "f32", f"f32mfma segments D={D} causal={causal}", ref="fact")


@pytest.mark.parametrize("tau", [1.0 / 32, 0.5])
def test_f32mfma_score_scale(tau):
    inp = make_inputs(1, 2, 300, 32, 9400, "f32")
    check(inp, True, "f32", f"f32mfma tau={tau}", scale=tau)


@pytest.mark.parametrize("name", ["small_noncausal_f32", "lra_causal_f32_p2"])
def test_f32mfma_workloads_full(name):
    w = WORKLOADS[name]
    inp = workload_inputs(w)
    check(inp, w.causal, w.dtype, f"{name} (every row)", ref="fact")


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("D,dtype", [(16, "f32"), (32, "bf16")])
def test_f32mfma_one_segment_per_head(D, dtype, causal):
    """Enough heads for one workgroup per (head, slice) (no segments, no
    workspace; at D <= 32 the plan aims at 512 workgroups, two per CU): the
    non-causal totals and queries in one launch, the causal scan from an
    empty state."""
    B, H = (16, 32) if D == 16 else (16, 16)
    assert fm.workspace_bytes(B, H, 100, D, 2, causal, fm.F32 if dtype == "f32" else fm.BF16) == 0
    inp = make_inputs(B, H, 100, D, 9500 + D, dtype)
    check(inp, causal, dtype, f"f32mfma one segment D={D} {dtype} causal={causal}")


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("BH", [(2, 4), (3, 4)])
def test_f32mfma_d128_one_segment(BH, dtype, causal):
    """D = 128 with one workgroup per (head, slice, quarter of the features):
    no segment sums, the workspace holds only the partial F and G."""
    B, H = BH
    N = 100
    ws = fm.workspace_bytes(B, H, N, 128, 2, causal, fm.F32 if dtype == "f32" else fm.BF16)
    r256 = lambda b: (b + 255) // 256 * 256
    assert ws == r256(B * H * 4 * N * 128 * 4) + r256(B * H * 4 * N * 4), ws
    inp = make_inputs(B, H, N, 128, 9600 + B, dtype)
    check(inp, causal, dtype, f"f32mfma D=128 one segment B={B} H={H} {dtype} causal={causal}")


# ---------------------------------------------------------------------------
# p = 1 (f = 1 + s: the linear tiles alone, G = n + q^.y2), every D and dtype.
# Weights change sign and G_i may nearly cancel, so O is held to its
# conditioning-scaled bar (gpu_util.row_scaled: |dO_ij| <= TOL kappa_i
# (1 + kappa_i) max|v|, kappa_i = sum_n |w_in| / |G_i|) and G to TOL times
# sum_n |w_in|.
# ---------------------------------------------------------------------------
def check_p1(inp, causal, dtype, label, scale=None):
    import torch
    from gpu_util import row_scaled
    q, k, v = (to_dev(inp[n], dtype) for n in ("q", "k", "v"))
    o, g = fm.fastmax_fwd(q, k, v, p=1, causal=causal, scale=scale)
    torch.cuda.synchronize()
    tau = 1.0 if scale is None else scale
    ro, rg, rabs = oracle.fwd_brute(inp["q64"], inp["k64"], inp["v64"], 1, causal,
                                    with_abs=True, scale=tau)
    out = to_f64(o)
    gg = g.cpu().numpy().astype(np.float64)
    assert np.isfinite(out).all() and np.isfinite(gg).all(), label
    e, nill = row_scaled(out, ro, rg, rabs, np.abs(inp["v64"]).max())
    eg = float((np.abs(gg - rg) / rabs).max())
    say(f"{label}: E_O/bound={e:.3e} E_G={eg:.3e} (rows with kappa > 10: {nill})")
    assert e <= TOL[dtype] and eg <= TOL[dtype], (label, e, eg)


P1_CASES = [(D, causal, dtype) for D in (16, 32, 64, 128) for causal in (False, True)
            for dtype in ("f32", "bf16")]
P1_SHAPES = [(1, 1, 1), (1, 2, 33), (2, 3, 100), (1, 1, 1000)]


@pytest.mark.parametrize("shape", P1_SHAPES, ids=[f"B{b}H{h}N{n}" for b, h, n in P1_SHAPES])
@pytest.mark.parametrize("case", P1_CASES, ids=[f"D{d}-{'causal' if c else 'noncausal'}-{t}" for d, c, t in P1_CASES])
def test_f32mfma_p1_vs_brute(case, shape):
    D, causal, dtype = case
    B, H, N = shape
    inp = make_inputs(B, H, N, D, 9150 + D + N + 7 * H, dtype)
    check_p1(inp, causal, dtype, f"f32mfma p=1 D={D} causal={causal} {dtype} B={B} H={H} N={N}")


@pytest.mark.parametrize("D", [16, 64, 128])
@pytest.mark.parametrize("causal", [False, True])
def test_f32mfma_p1_many_segments(D, causal):
    """One head of 4000 tokens split into segments (p = 1)."""
    inp = make_inputs(1, 1, 4000, D, 9350 + D, "f32")
    check_p1(inp, causal, "f32", f"f32mfma p=1 segments D={D} causal={causal}")


def test_f32mfma_p1_scale_and_lra_workload():
    """The LRA-shaped p = 1 workload (B2 H4 N2048 D32, causal, f32) on every
    row, and a scaled call (tau = 1/32)."""
    w = WORKLOADS["lra_causal_f32_p1"]
    inp = workload_inputs(w)
    check_p1(inp, w.causal, w.dtype, f"{w.name} (every row)")
    inp = make_inputs(1, 2, 300, 32, 9450, "f32")
    check_p1(inp, True, "f32", "f32mfma p=1 tau=1/32", scale=1.0 / 32)

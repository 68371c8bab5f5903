"""GPU parity of the score-scaled entry points (weights f_p(tau q^.k^)).

Every kernel path -- the generic float32 VALU kernels, the MFMA causal scan,
the MFMA non-causal path, and the MFMA and generic backward -- is compared
with the fp64 oracle run at the same tau, for tau = 1/D (the unit-norm
variant) and tau = 1/sqrt(D) (softmax's temperature), at the tolerances of
the other parity tests.  tau = 1 through the scaled calls must reproduce the
unscaled calls bit for bit on the MFMA paths (the generic kernels, whose
partial sums meet in atomics, to within their run-to-run rounding).
"""
import math

import numpy as np
import pytest

import oracle
from paper_2402_07901_amd import fastmax as fm
from paper_2402_07901_amd.inputs import make_inputs

from gpu_util import TOL, max_rel, row_scaled, say, to_dev, to_f64

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fm.lib()
    yield
    torch.cuda.synchronize()


def taus(D):
    return (1.0 / D, 1.0 / math.sqrt(D))


def fwd_check(inp, p, causal, dtype, tau, label):
    import torch
    q, k, v = (to_dev(inp[n], dtype) for n in ("q", "k", "v"))
    o, g = fm.fastmax_fwd(q, k, v, p=p, causal=causal, scale=tau)
    torch.cuda.synchronize()
    ref_o, ref_g, ref_gabs = oracle.fwd_brute(inp["q64"], inp["k64"], inp["v64"], p, causal,
                                              with_abs=True, scale=tau)
    out = to_f64(o)
    gg = g.cpu().numpy().astype(np.float64)
    assert np.isfinite(out).all(), label
    if p == 2:
        e = max_rel(out, ref_o)
        eg = float((np.abs(gg - ref_g) / np.abs(ref_g)).max())
    else:
        e, _ = row_scaled(out, ref_o, ref_g, ref_gabs, np.abs(inp["v64"]).max())
        eg = float((np.abs(gg - ref_g) / ref_gabs).max())
    say(f"{label} tau={tau:.4g}: E_O={e:.3e} E_G={eg:.3e}")
    assert e <= TOL[dtype], (label, tau, e)
    assert eg <= TOL[dtype], (label, tau, eg)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("p", [1, 2])
@pytest.mark.parametrize("D", [16, 32, 64])
def test_fwd_scaled_generic(D, p, causal, dtype):
    """Generic kernels (every case except D = 64, p = 2, bf16 with N >= 128
    non-causal or any N causal)."""
    N = 100 if not (D == 64 and p == 2 and dtype == "bf16" and causal) else 17
    label = f"fwd scaled N={N} D={D} p={p} causal={causal} {dtype}"
    say(label)
    inp = make_inputs(2, 2, N, D, 700 + D + N, dtype)
    for tau in taus(D):
        fwd_check(inp, p, causal, dtype, tau, label)


@pytest.mark.parametrize("N", [300, 1000])
def test_fwd_scaled_mfma_causal(N):
    label = f"fwd scaled MFMA causal N={N}"
    say(label)
    inp = make_inputs(1, 3, N, 64, 710 + N, "bf16")
    for tau in taus(64):
        fwd_check(inp, 2, True, "bf16", tau, label)


@pytest.mark.parametrize("N", [128, 1000])
def test_fwd_scaled_mfma_noncausal(N):
    label = f"fwd scaled MFMA non-causal N={N}"
    say(label)
    inp = make_inputs(1, 3, N, 64, 720 + N, "bf16")
    for tau in taus(64):
        fwd_check(inp, 2, False, "bf16", tau, label)


def bwd_check(inp, p, causal, dtype, tau, label):
    import torch
    q, k, v = (to_dev(inp[n], dtype) for n in ("q", "k", "v"))
    do = to_dev(inp["dout"], dtype)
    o, g = fm.fastmax_fwd(q, k, v, p=p, causal=causal, scale=tau)
    dq, dk, dv = fm.fastmax_bwd(q, k, v, o, do, g, p=p, causal=causal, scale=tau)
    torch.cuda.synchronize()
    rq, rk, rv = oracle.bwd_brute(inp["q64"], inp["k64"], inp["v64"], inp["dout64"], p, causal,
                                  scale=tau)
    for nm, got, ref in (("dq", dq, rq), ("dk", dk, rk), ("dv", dv, rv)):
        x = to_f64(got)
        e = max_rel(x, ref)
        say(f"{label} tau={tau:.4g} {nm}: E={e:.3e}")
        assert np.isfinite(x).all()
        assert e <= TOL[dtype], (label, tau, nm, e)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("p", [1, 2])
@pytest.mark.parametrize("D", [16, 64])
def test_bwd_scaled_generic(D, p, causal, dtype):
    """At tau = 1/D every p = 1 weight 1 + tau s is >= 0 (|tau s| <= 1), so
    kappa = 1 and the plain tensor-wide bar pins the p = 1 backward in both
    I/O dtypes (with bf16 I/O, D = 64, p = 2 this is the MFMA backward when
    causal)."""
    label = f"bwd scaled generic D={D} p={p} causal={causal} {dtype}"
    say(label)
    inp = make_inputs(1, 2, 37, D, 730 + D, dtype, with_dout=True)
    for tau in taus(D):
        bwd_check(inp, p, causal, dtype, tau, label)


@pytest.mark.parametrize("N", [300])
def test_bwd_scaled_mfma_noncausal(N):
    label = f"bwd scaled MFMA non-causal N={N} bf16"
    say(label)
    inp = make_inputs(1, 2, N, 64, 760 + N, "bf16", with_dout=True)
    for tau in taus(64):
        bwd_check(inp, 2, False, "bf16", tau, label)


@pytest.mark.parametrize("N", [37, 300])
def test_bwd_scaled_mfma_causal(N):
    label = f"bwd scaled MFMA causal N={N} bf16"
    say(label)
    inp = make_inputs(1, 2, N, 64, 740 + N, "bf16", with_dout=True)
    for tau in taus(64):
        bwd_check(inp, 2, True, "bf16", tau, label)


@pytest.mark.parametrize("case", [(300, 64, 2, True, "bf16"), (300, 64, 2, False, "bf16"),
                                  (50, 32, 2, True, "f32"), (50, 16, 1, False, "bf16")])
def test_scale_one_is_the_unscaled_call(case):
    import torch
    N, D, p, causal, dtype = case
    say(f"tau = 1 identity {case}")
    inp = make_inputs(1, 2, N, D, 750 + N, dtype, with_dout=True)
    q, k, v = (to_dev(inp[n], dtype) for n in ("q", "k", "v"))
    do = to_dev(inp["dout"], dtype)
    o0, g0 = fm.fastmax_fwd(q, k, v, p=p, causal=causal)
    o1, g1 = fm.fastmax_fwd(q, k, v, p=p, causal=causal, scale=1.0)
    d0 = fm.fastmax_bwd(q, k, v, o0, do, g0, p=p, causal=causal)
    d1 = fm.fastmax_bwd(q, k, v, o0, do, g0, p=p, causal=causal, scale=1.0)
    torch.cuda.synchronize()
    # The MFMA kernels are deterministic: bit-identical.  The generic kernels
    # meet partial sums in atomics (LDS in the forward's contraction, fp32
    # global atomics across slices in the backward), so two runs differ by
    # summation order: bounded relative to the tensor's largest entry
    # (cancellation makes small entries differ by more than their own ulp).
    mfma_fwd = D == 64 and p == 2 and dtype == "bf16" and (causal or N >= 128)
    mfma_bwd = D == 64 and p == 2 and dtype == "bf16" and causal
    bound = 2.0 ** -8 if dtype == "bf16" else 2e-5

    def same(a, b, exact, what):
        if exact:
            assert torch.equal(a, b), what
        else:
            e = max_rel(to_f64(a), to_f64(b))
            say(f"  {what}: generic run-to-run E={e:.3e}")
            assert e <= bound, (what, e)

    same(o0, o1, mfma_fwd, "O")
    same(g0, g1, mfma_fwd, "G")
    for nm, a, b in zip(("dq", "dk", "dv"), d0, d1):
        same(a, b, mfma_bwd, nm)

"""GPU tests of the two-segment split of the causal MFMA scans (the forward
and the backward's dv scan; fastmax_set_scan_segments).

The first workgroup of a split (head, slice) scans the chunks before the
split and emits its summary (moment state, Y3, y2, x1: the exclusive prefix
of Sec. 2.4's causal recurrences at the split); the second starts from it,
or (REBUILD, and after a timed-out wait) rebuilds that prefix itself.  Both
perform the unsplit scan's operations in the same order, so every mode must
give bit-identical O, G, dq, dk, dv; the split results are also held to the
fp64 oracle (explicit N x N definition, Sec. 2.2) at the bf16 bar.  Shapes
cover 2, 3 (odd: split after 1 chunk), 4, 6 and 8 chunks with ragged last
chunks, a single chunk (never split), and the B8 H12 N4096 shape where the
automatic plan splits (384 scans on 256 CUs).
"""
import numpy as np
import pytest

import oracle
from paper_2402_07901_amd import fastmax as fm
from paper_2402_07901_amd.inputs import WORKLOADS, make_inputs, workload_inputs

from gpu_util import TOL, max_rel, say, to_dev, to_f64

pytestmark = pytest.mark.gpu

MODES = {"off": fm.SCAN_SEGMENTS_OFF, "on": fm.SCAN_SEGMENTS_ON,
         "rebuild": fm.SCAN_SEGMENTS_REBUILD, "auto": fm.SCAN_SEGMENTS_AUTO}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fm.lib()
    prev = fm.set_scan_segments(fm.SCAN_SEGMENTS_AUTO)
    yield
    fm.set_scan_segments(prev)
    torch.cuda.synchronize()


def fwd_all_modes(q, k, v):
    import torch
    res = {}
    for name, mode in MODES.items():
        fm.set_scan_segments(mode)
        o, g = fm.fastmax_fwd(q, k, v, p=2, causal=True)
        torch.cuda.synchronize()
        res[name] = (o, g)
    fm.set_scan_segments(fm.SCAN_SEGMENTS_AUTO)
    return res


def assert_same(res, label):
    import torch
    o0, g0 = res["off"]
    for name, (o, g) in res.items():
        assert torch.equal(o.view(torch.int16), o0.view(torch.int16)), (label, name)
        assert torch.equal(g, g0), (label, name)


FWD_SHAPES = [(1, 1, 256), (1, 2, 129), (1, 1, 384), (2, 3, 385), (3, 5, 700), (1, 1, 1000),
              (1, 1, 128)]


@pytest.mark.parametrize("shape", FWD_SHAPES, ids=[f"B{b}H{h}N{n}" for b, h, n in FWD_SHAPES])
def test_forward_modes_bit_identical_and_vs_brute(shape):
    B, H, N = shape
    say(f"segments forward B={B} H={H} N={N}")
    inp = make_inputs(B, H, N, 64, 7100 + N + H, "bf16")
    q, k, v = (to_dev(inp[n], "bf16") for n in ("q", "k", "v"))
    res = fwd_all_modes(q, k, v)
    assert_same(res, shape)
    ref_o, ref_g = oracle.fwd_brute(inp["q64"], inp["k64"], inp["v64"], 2, True)
    o, g = res["on"]
    e = max_rel(to_f64(o), ref_o)
    gg = g.cpu().numpy().astype(np.float64)
    eg = float((np.abs(gg - ref_g) / np.abs(ref_g)).max())
    say(f"segments forward {shape}: split vs brute E_O={e:.3e} E_G={eg:.3e}")
    assert e <= TOL["bf16"] and eg <= TOL["bf16"], (shape, e, eg)


BWD_SHAPES = [(1, 2, 300), (2, 2, 1000)]


@pytest.mark.parametrize("shape", BWD_SHAPES, ids=[f"B{b}H{h}N{n}" for b, h, n in BWD_SHAPES])
def test_backward_modes_bit_identical(shape):
    import torch
    B, H, N = shape
    say(f"segments backward B={B} H={H} N={N}")
    inp = make_inputs(B, H, N, 64, 7300 + N, "bf16", with_dout=True)
    q, k, v, do = (to_dev(inp[n], "bf16") for n in ("q", "k", "v", "dout"))
    fm.set_scan_segments(fm.SCAN_SEGMENTS_OFF)
    o, g = fm.fastmax_fwd(q, k, v, p=2, causal=True)
    ref = fm.fastmax_bwd(q, k, v, o, do, g, p=2, causal=True)
    torch.cuda.synchronize()
    for name, mode in MODES.items():
        fm.set_scan_segments(mode)
        got = fm.fastmax_bwd(q, k, v, o, do, g, p=2, causal=True)
        torch.cuda.synchronize()
        for a, b_, what in zip(got, ref, ("dq", "dk", "dv")):
            assert torch.equal(a.view(torch.int16), b_.view(torch.int16)), (shape, name, what)
    fm.set_scan_segments(fm.SCAN_SEGMENTS_AUTO)
    # the split backward against the fp64 explicit backward
    from test_parity_gpu import bwd_case
    fm.set_scan_segments(fm.SCAN_SEGMENTS_ON)
    try:
        bwd_case(inp, 2, True, "bf16", label=f"segments bwd {shape}")
    finally:
        fm.set_scan_segments(fm.SCAN_SEGMENTS_AUTO)


def test_full_shape_auto_split_matches_unsplit():
    """B8 H12 N4096 (the forward+backward workload's shape): the automatic
    plan splits the forward's scans (384 on 256 CUs); forward and backward
    (its dv scan split under ON) are bit-identical to the unsplit scans, and
    the rebuilt prefixes give the same forward."""
    import torch
    w = WORKLOADS["fwdbwd_causal_bf16"]
    say(f"{w.name}: auto (split) vs off vs rebuild")
    inp = workload_inputs(w)
    q, k, v, do = (to_dev(inp[n], "bf16") for n in ("q", "k", "v", "dout"))
    res = fwd_all_modes(q, k, v)
    assert_same(res, w.name)
    o, g = res["off"]
    grads = {}
    for name in ("off", "on", "auto"):
        fm.set_scan_segments(MODES[name])
        grads[name] = fm.fastmax_bwd(q, k, v, o, do, g, p=2, causal=True)
        torch.cuda.synchronize()
    fm.set_scan_segments(fm.SCAN_SEGMENTS_AUTO)
    for name in ("on", "auto"):
        for a, b_, what in zip(grads[name], grads["off"], ("dq", "dk", "dv")):
            assert torch.equal(a.view(torch.int16), b_.view(torch.int16)), (name, what)

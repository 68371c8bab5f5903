"""GPU test of the allocation-free forward (fastmax_fwd_noalloc).

Called through the C ABI on two problems in a row, the second smaller than
the first (the per-GPU scratch keeps the first call's contents), on each
forward path: the causal and non-causal MFMA kernels (bf16, D = 64, p = 2;
deterministic, so bit-identical to fastmax_fwd) and the float32 kernels
(their partial sums meet in atomics: equal to fastmax_fwd within run-to-run
rounding).  Also checked against the fp64 oracle at the bf16 / f32 bars.
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


CASES = [
    # (label, D, p, causal, dtype, first shape, second (smaller) shape)
    ("causal MFMA", 64, 2, True, "bf16", (2, 4, 3000), (1, 3, 700)),
    ("non-causal MFMA", 64, 2, False, "bf16", (1, 2, 5000), (1, 1, 1000)),
    ("float32 kernels", 32, 2, True, "f32", (1, 2, 2000), (1, 1, 300)),
    ("float32 kernels p = 1", 16, 1, False, "bf16", (1, 1, 4000), (1, 1, 257)),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_noalloc_matches_fastmax_fwd_twice(case):
    import torch
    label, D, p, causal, dtype, s1, s2 = case
    exact = D == 64 and p == 2 and dtype == "bf16"
    for call, (B, H, N) in enumerate((s1, s2)):
        say(f"{label}: call {call + 1}, B={B} H={H} N={N}")
        need = fm.workspace_bytes(B, H, N, D, p, causal, fm.BF16 if dtype == "bf16" else fm.F32)
        assert need <= fm.NOALLOC_MAX_WORKSPACE_BYTES
        inp = make_inputs(B, H, N, D, 1200 + 10 * call + D, dtype)
        q, k, v = (to_dev(inp[n], dtype) for n in ("q", "k", "v"))
        o_ref, g_ref = fm.fastmax_fwd(q, k, v, p=p, causal=causal)
        out = torch.empty_like(q)
        g = torch.empty((B, H, N), dtype=torch.float32, device=q.device)
        fm.fastmax_fwd_noalloc(q, k, v, out, g, p=p, causal=causal)
        torch.cuda.synchronize()
        if exact:
            assert torch.equal(out.view(torch.int16), o_ref.view(torch.int16)), label
            assert torch.equal(g, g_ref), label
        else:
            bound = 2.0 ** -8 if dtype == "bf16" else 2e-5
            e = max_rel(to_f64(out), to_f64(o_ref))
            eg = max_rel(to_f64(g), to_f64(g_ref))
            say(f"{label}: vs fastmax_fwd E_O={e:.3e} E_G={eg:.3e}")
            assert e <= bound and eg <= bound, (label, e, eg)
        ro, rg = oracle.fwd_fact(inp["q64"], inp["k64"], inp["v64"], p, causal)
        if p == 2:
            e = max_rel(to_f64(out), ro)
            say(f"{label}: vs oracle E_O={e:.3e}")
            assert e <= TOL[dtype], (label, e)


def test_noalloc_rejects_beyond_scratch_on_device():
    """A forward whose workspace exceeds the scratch is refused with
    EWORKSPACE and leaves the output untouched."""
    import torch
    B, H, N, D = 1, 1, 300000, 64
    assert fm.workspace_bytes(B, H, N, D, 2, 1, fm.BF16) > fm.NOALLOC_MAX_WORKSPACE_BYTES
    q = torch.zeros((B, H, N, D), dtype=torch.bfloat16, device="cuda")
    out = torch.full_like(q, 3.0)
    rc = fm.fastmax_fwd_noalloc_raw(q, q, q, out, None, B, H, N, D, 2, True, fm.BF16, None)
    torch.cuda.synchronize()
    assert rc == fm.EWORKSPACE
    assert bool((out == 3.0).all())

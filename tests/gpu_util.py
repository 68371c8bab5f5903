"""Helpers for the GPU parity tests: device transfer and error metrics."""
import sys

import numpy as np

from paper_2402_07901_amd.inputs import bf16_bits_to_f64


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_dev(arr, dtype):
    import torch
    if dtype == "f32":
        return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).cuda()
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(arr, dtype=np.uint16).view(np.int16))
        return t.cuda().view(torch.bfloat16)
    raise ValueError(dtype)


def to_f64(t):
    import torch
    if t.dtype == torch.bfloat16:
        return bf16_bits_to_f64(t.view(torch.int16).cpu().numpy().view(np.uint16))
    return t.detach().cpu().numpy().astype(np.float64)


TOL = {"f32": 1e-4, "bf16": 2e-2}


def max_rel(x, ref):
    """max|x - ref| / max|ref| (the tensor-wide relative error)."""
    den = np.abs(ref).max()
    return float(np.abs(x - ref).max() / (den if den > 0 else 1.0))


def row_scaled(x, ref, g_ref, gabs_ref, vmax):
    """Per-row error scaled by the row's conditioning.

    O_i = F_i / G_i with |dF_i| <~ eps sum_n |w_in||v_n| <= eps kappa_i |G_i| max|v|
    and |dG_i| <~ eps kappa_i |G_i|, kappa_i = sum_n |w_in| / |G_i|; to first
    order |dO_ij| <= eps kappa_i (1 + kappa_i) max|v| (|O_ij| <= kappa_i max|v|).
    Returns (max_i max_j |x_ij - ref_ij| / (kappa_i (1 + kappa_i) max|v|),
    number of rows with kappa_i > 10)."""
    kappa = gabs_ref / np.abs(g_ref)
    e = np.abs(x - ref).max(-1) / (kappa * (1.0 + kappa) * vmax)
    return float(e.max()), int((kappa > 10).sum())

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


def grad_bounds(q64, k64, v64, dout64, o_ref, g_ref, gabs_ref, p, causal, tau=1.0):
    """First-order rounding bounds of the gradient entries of ONE head
    ([N, D] arrays), for conditioning-aware comparisons (p = 1, where
    weights change sign and G_i may nearly cancel).

    The gradient is a sum over (query i, key n) of terms that each carry
    1/G_i, O_i and f'(tau s_in); a relative rounding error eps in the
    forward's sums gives G_i a relative error ~ eps kappa_i
    (kappa_i = sum_n |w_in| / |G_i|) and O_i an absolute error
    ~ eps kappa_i (1 + kappa_i) max|v|, so each term (i, n) has an error of
    about eps kappa_i times its magnitude
        A_in = |f'(tau s_in)| |dO_i|_1 max|v| (1 + kappa_i) / |G_i|.
    Summed without cancellation, and carried through the standardisation
    backward (|d x| <= (2 + max|x^|) |d x^| / sigma), this gives per row i
    of dq, and per key n of dk and dv, a bound B such that
    |error| <= eps B.  Returns (Bq [N], Bk [N], Bv [N])."""
    import oracle
    qh, _, sq = oracle.standardize(q64)
    kh, _, sk = oracle.standardize(k64)
    N = q64.shape[0]
    s = tau * (qh @ kh.T)
    w = 1.0 + s + (0.5 * s * s if p == 2 else 0.0)
    dw = np.ones_like(s) if p == 1 else 1.0 + s
    if causal:
        mask = np.tril(np.ones((N, N), dtype=bool))
        w = np.where(mask, w, 0.0)
        dw = np.where(mask, dw, 0.0)
    kappa = gabs_ref / np.abs(g_ref)
    vmax = np.abs(v64).max()
    a_row = np.abs(dout64).sum(-1) * vmax * (1.0 + kappa) / np.abs(g_ref)   # [N] over i
    A = np.abs(dw) * (kappa * a_row)[:, None]                               # [i, n]
    bq_hat = tau * (A @ np.abs(kh)).max(-1)                                 # [i]
    bk_hat = tau * (A.T @ np.abs(qh)).max(-1)                               # [n]
    Bq = (2.0 + np.abs(qh).max(-1)) * bq_hat / sq
    Bk = (2.0 + np.abs(kh).max(-1)) * bk_hat / sk
    Bv = (np.abs(w) * (kappa * np.abs(dout64).max(-1) / np.abs(g_ref))[:, None]).sum(0)
    return Bq, Bk, Bv


def bounded_err(x, ref, bound):
    """max over rows r of max_j |x_rj - ref_rj| / bound_r."""
    return float((np.abs(x - ref).max(-1) / bound).max())

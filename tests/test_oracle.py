"""Pins for the fp64 oracle (CPU only).

Each check ties the oracle to something other than itself: hand-derived
golden values (tests/golden), a library matmul of the explicit attention
matrix, closed forms, invariants the paper states, central finite
differences and PyTorch float64 autograd.  A final test plants plausible
mistakes into copies of the oracle source and shows that the pins catch each.
"""
import json
import math
import os
import shutil
import subprocess
from fractions import Fraction

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _frac(x):
    if isinstance(x, str):
        return float(Fraction(x))
    return float(x)


def _arr(a):
    return np.array([[_frac(x) for x in row] for row in a]) if isinstance(a[0], list) \
        else np.array([_frac(x) for x in a])


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _rand(B, H, N, D, seed):
    rng = np.random.default_rng([2402, 7901, 1000 + seed])
    return (rng.standard_normal((B, H, N, D)), rng.standard_normal((B, H, N, D)),
            rng.standard_normal((B, H, N, D)))


# --------------------------------------------------------------------------
# checks (raise AssertionError); shared with the planted-mistake test
# --------------------------------------------------------------------------
def check_golden_standardize():
    g = _load("standardize_d2_d3.json")
    for c in g["cases"]:
        x = np.array(c["x"], dtype=np.float64)[None]
        xh, mu, sg = oracle.standardize(x)
        np.testing.assert_allclose(xh[0], [_frac(t) for t in c["xhat"]], rtol=0, atol=1e-13)
        np.testing.assert_allclose(mu[0], _frac(c["mean"]), rtol=0, atol=1e-14)
        np.testing.assert_allclose(sg[0], _frac(c["std"]), rtol=1e-13)


def _golden_forward_cases(name):
    g = _load(name)
    q = np.array(g["q"], dtype=np.float64)[None, None]
    k = np.array(g["k"], dtype=np.float64)[None, None]
    v = np.array(g["v"], dtype=np.float64)[None, None]
    for c in g["cases"]:
        yield q, k, v, c["p"], c["causal"], _arr(c["O"]), _arr(c["G"])


def check_golden_forward():
    for name in ("forward_d2_n2.json", "forward_d4_n3.json"):
        for q, k, v, p, causal, O, G in _golden_forward_cases(name):
            for fn in (oracle.fwd_brute, oracle.fwd_fact):
                o, g = fn(q, k, v, p, causal)
                np.testing.assert_allclose(o[0, 0], O, rtol=0, atol=1e-12)
                np.testing.assert_allclose(g[0, 0], G, rtol=1e-13)
            N = q.shape[2]
            o, g = oracle.fwd_rows(q, k, v, p, causal, np.arange(N))
            np.testing.assert_allclose(o, O, rtol=0, atol=1e-12)
            A = oracle.attention_matrix(q[0, 0], k[0, 0], p, causal)
            np.testing.assert_allclose(A @ v[0, 0], O, rtol=0, atol=1e-12)


def check_golden_backward():
    g = _load("backward_d2_n2.json")
    q = np.array(g["q"], dtype=np.float64)[None, None]
    k = np.array(g["k"], dtype=np.float64)[None, None]
    v = np.array(g["v"], dtype=np.float64)[None, None]
    do = np.array(g["dout"], dtype=np.float64)[None, None]
    for c in g["cases"]:
        dq, dk, dv = oracle.bwd_brute(q, k, v, do, c["p"], c["causal"])
        np.testing.assert_allclose(dv[0, 0], _arr(c["dv"]), rtol=0, atol=1e-12)
        np.testing.assert_allclose(dq[0, 0], _arr(c["dq"]), rtol=0, atol=1e-12)
        np.testing.assert_allclose(dk[0, 0], _arr(c["dk"]), rtol=0, atol=1e-12)


def check_brute_vs_fact(shapes=((1, 2, 37, 4), (2, 1, 64, 8), (1, 1, 33, 16))):
    for si, (B, H, N, D) in enumerate(shapes):
        q, k, v = _rand(B, H, N, D, si)
        for p in (1, 2):
            for causal in (False, True):
                ob, gb = oracle.fwd_brute(q, k, v, p, causal)
                of, gf = oracle.fwd_fact(q, k, v, p, causal)
                # p = 1 weights 1 + s change sign (|s| reaches D under Eq. 7),
                # so G may nearly cancel: compare absolutely with a looser bound.
                scale = np.abs(ob).max() if p == 2 else 1.0
                tol = 1e-11 if p == 2 else 1e-8
                err = np.abs(ob - of).max() / scale
                assert err < tol, (B, H, N, D, p, causal, err)
                np.testing.assert_allclose(gb, gf, rtol=1e-10, atol=1e-9)


def _fd_grads(q, k, v, do, p, causal, h=1e-6, scale=1.0):
    def loss(q_, k_, v_):
        o, _ = oracle.fwd_brute(q_, k_, v_, p, causal, scale=scale)
        return float((o * do).sum())
    grads = []
    for which in range(3):
        base = [q.copy(), k.copy(), v.copy()]
        gr = np.zeros_like(q)
        it = np.nditer(q, flags=["multi_index"])
        for _ in it:
            idx = it.multi_index
            plus = [a.copy() for a in base]
            minus = [a.copy() for a in base]
            plus[which][idx] += h
            minus[which][idx] -= h
            gr[idx] = (loss(*plus) - loss(*minus)) / (2 * h)
        grads.append(gr)
    return grads


def check_bwd_finite_differences():
    for p in (1, 2):
        for causal in (False, True):
            q, k, v = _rand(1, 1, 5, 4, 7 + p)
            do = np.random.default_rng([2402, 7901, 77]).standard_normal(q.shape)
            dq, dk, dv = oracle.bwd_brute(q, k, v, do, p, causal)
            fq, fk, fv = _fd_grads(q, k, v, do, p, causal)
            for a, b, nm in ((dq, fq, "dq"), (dk, fk, "dk"), (dv, fv, "dv")):
                err = np.abs(a - b).max() / max(1.0, np.abs(b).max())
                assert err < 2e-6, (nm, p, causal, err)


def _std_np(x):
    c = x - x.mean(-1, keepdims=True)
    return c / np.sqrt((c ** 2).mean(-1, keepdims=True))


# Score scale tau (weights f_p(tau s); tau = 1/D is the unit-norm variant,
# Sec. 2.3 assumes |s| <= 1).
def check_scale_p1_closed_form():
    """p = 1: w = 1 + tau s, so o_i = (sum v + tau (sum v k^T) q^_i) /
    (n_i + tau q^_i . sum k^), on both oracle routes."""
    q, k, v = _rand(1, 1, 25, 6, 31)
    qh, kh, vv = _std_np(q)[0, 0], _std_np(k)[0, 0], v[0, 0]
    tau = 1.0 / 6
    for causal in (False, True):
        exp = np.empty((25, 6))
        for i in range(25):
            n = i + 1 if causal else 25
            exp[i] = (vv[:n].sum(0) + tau * (vv[:n].T @ kh[:n]) @ qh[i]) / \
                (n + tau * qh[i] @ kh[:n].sum(0))
        for route in (oracle.fwd_brute, oracle.fwd_fact):
            o, _ = route(q, k, v, 1, causal, scale=tau)
            np.testing.assert_allclose(o[0, 0], exp, rtol=1e-10, atol=1e-10)


def check_scale_p2_explicit():
    """p = 2 on a tiny problem: W = 1 + tau S + (tau S)^2 / 2 written out."""
    q, k, v = _rand(1, 1, 9, 4, 33)
    qh, kh, vv = _std_np(q)[0, 0], _std_np(k)[0, 0], v[0, 0]
    tau = 0.37
    S = tau * (qh @ kh.T)
    W = 1 + S + S * S / 2
    for causal in (False, True):
        Wc = np.tril(W) if causal else W
        exp, gexp = (Wc @ vv) / Wc.sum(1, keepdims=True), Wc.sum(1)
        for route in (oracle.fwd_brute, oracle.fwd_fact):
            o, g = route(q, k, v, 2, causal, scale=tau)
            np.testing.assert_allclose(o[0, 0], exp, rtol=1e-11, atol=1e-11)
            np.testing.assert_allclose(g[0, 0], gexp, rtol=1e-11)


def check_scale_small_limit():
    """tau -> 0: every weight tends to 1, O_i to the mean of the visible values."""
    q, k, v = _rand(1, 2, 30, 8, 32)
    pref = np.cumsum(v, 2) / np.arange(1, 31)[:, None]
    for p in (1, 2):
        for causal in (False, True):
            exp = pref if causal else np.broadcast_to(v.mean(2, keepdims=True), v.shape)
            for route in (oracle.fwd_brute, oracle.fwd_fact):
                o, _ = route(q, k, v, p, causal, scale=1e-9)
                np.testing.assert_allclose(o, exp, atol=1e-6)


def check_scale_bwd_finite_differences():
    for p in (1, 2):
        for causal in (False, True):
            q, k, v = _rand(1, 1, 5, 4, 40 + p)
            do = np.random.default_rng([2402, 7901, 78]).standard_normal(q.shape)
            dq, dk, dv = oracle.bwd_brute(q, k, v, do, p, causal, scale=0.3)
            fq, fk, fv = _fd_grads(q, k, v, do, p, causal, scale=0.3)
            for a, b, nm in ((dq, fq, "dq"), (dk, fk, "dk"), (dv, fv, "dv")):
                err = np.abs(a - b).max() / max(1.0, np.abs(b).max())
                assert err < 2e-6, (nm, p, causal, err)


# --------------------------------------------------------------------------
# pytest entry points
# --------------------------------------------------------------------------
def test_scale_p1_closed_form():
    check_scale_p1_closed_form()


def test_scale_p2_explicit():
    check_scale_p2_explicit()


def test_scale_small_limit():
    check_scale_small_limit()


def test_scale_bwd_finite_differences():
    check_scale_bwd_finite_differences()


@pytest.mark.parametrize("causal", [False, True])
def test_unit_norm_makes_p1_weights_valid(causal):
    """With tau = 1/D, |tau s| <= 1, so f_1 = 1 + tau s >= 0 and the rows of A
    are convex weights (Eq. "valid"); with tau = 1 some weights are negative
    on the same inputs."""
    q, k, _ = _rand(1, 1, 64, 8, 34)
    A = oracle.attention_matrix(q[0, 0], k[0, 0], 1, causal, scale=1.0 / 8)
    assert A.min() >= 0.0
    np.testing.assert_allclose(A.sum(1), 1.0, rtol=1e-12)
    A1 = oracle.attention_matrix(q[0, 0], k[0, 0], 1, causal)
    assert A1.min() < 0.0
def test_golden_standardize():
    check_golden_standardize()


def test_standardize_invariants():
    x = np.random.default_rng(3).standard_normal((50, 64)) * 3 + 1.5
    xh, mu, sg = oracle.standardize(x)
    np.testing.assert_allclose(xh.sum(-1), 0, atol=1e-12)
    np.testing.assert_allclose((xh ** 2).sum(-1), 64, rtol=1e-13)
    np.testing.assert_allclose(mu, x.mean(-1), rtol=1e-13)
    np.testing.assert_allclose(sg, x.std(-1), rtol=1e-13)   # numpy std: ddof=0


def test_golden_forward():
    check_golden_forward()


def test_golden_backward():
    check_golden_backward()


def test_brute_vs_factorised():
    check_brute_vs_fact()


@pytest.mark.parametrize("p", [1, 2])
@pytest.mark.parametrize("causal", [False, True])
def test_explicit_matrix_rows_and_matmul(p, causal):
    q, k, v = _rand(1, 1, 48, 8, 11)
    A = oracle.attention_matrix(q[0, 0], k[0, 0], p, causal)
    np.testing.assert_allclose(A.sum(1), 1.0, atol=1e-12)          # Eq. valid
    if causal:
        assert np.all(np.triu(A, 1) == 0.0)
    if p == 2:
        assert np.all(A >= 0)
    o, _ = oracle.fwd_brute(q, k, v, p, causal)
    np.testing.assert_allclose(A @ v[0, 0], o[0, 0], rtol=1e-10, atol=1e-10)


@pytest.mark.parametrize("causal", [False, True])
def test_row_normalisation_invariants(causal):
    q, k, v = _rand(1, 2, 40, 8, 12)
    for fn in (oracle.fwd_brute, oracle.fwd_fact):
        o, _ = fn(q, k, np.ones_like(v), 2, causal)
        np.testing.assert_allclose(o, 1.0, atol=1e-12)
        c = np.broadcast_to(np.arange(8.0) - 3.0, v.shape).copy()
        o, _ = fn(q, k, c, 2, causal)
        np.testing.assert_allclose(o, c, atol=1e-11)


def test_p2_denominator_bound():
    q, k, v = _rand(2, 2, 64, 16, 13)
    _, g = oracle.fwd_fact(q, k, v, 2, False)
    assert np.all(g >= 64 / 2)                    # f_2 >= 1/2 for every pair
    _, g = oracle.fwd_fact(q, k, v, 2, True)
    i = np.arange(1, 65)
    assert np.all(g >= i / 2)


@pytest.mark.parametrize("p", [1, 2])
def test_causality(p):
    q, k, v = _rand(1, 1, 30, 8, 14)
    o, _ = oracle.fwd_fact(q, k, v, p, True)
    np.testing.assert_allclose(o[0, 0, 0], v[0, 0, 0], rtol=1e-14, atol=1e-14)  # O_1 = v_1
    for cut in (1, 10, 29):
        q2, k2, v2 = q.copy(), k.copy(), v.copy()
        rng = np.random.default_rng(cut)
        q2[:, :, cut:] = rng.standard_normal(q2[:, :, cut:].shape)
        k2[:, :, cut:] = rng.standard_normal(k2[:, :, cut:].shape)
        v2[:, :, cut:] = rng.standard_normal(v2[:, :, cut:].shape)
        for fn in (oracle.fwd_fact, oracle.fwd_brute):
            a, _ = fn(q, k, v, p, True)
            b, _ = fn(q2, k2, v2, p, True)
            np.testing.assert_array_equal(a[:, :, :cut], b[:, :, :cut])
        # a prefix is an exact sub-problem
        a, _ = oracle.fwd_brute(q[:, :, :cut], k[:, :, :cut], v[:, :, :cut], p, True)
        np.testing.assert_allclose(a, o[:, :, :cut], rtol=0, atol=1e-10)


def test_special_cases():
    q, k, v = _rand(1, 1, 1, 8, 15)
    for causal in (False, True):
        for p in (1, 2):
            o, _ = oracle.fwd_fact(q, k, v, p, causal)
            np.testing.assert_allclose(o, v, atol=1e-13)          # N = 1
    q, k, v = _rand(1, 1, 20, 8, 16)
    k[:] = k[:, :, :1]                                             # all keys equal
    o, _ = oracle.fwd_fact(q, k, v, 2, False)
    np.testing.assert_allclose(o[0, 0], np.broadcast_to(v[0, 0].mean(0), (20, 8)), atol=1e-12)
    o, _ = oracle.fwd_fact(q, k, v, 2, True)
    pref = np.cumsum(v[0, 0], 0) / np.arange(1, 21)[:, None]
    np.testing.assert_allclose(o[0, 0], pref, atol=1e-12)


def test_scale_shift_invariance():
    q, k, v = _rand(1, 2, 32, 16, 17)
    o0, _ = oracle.fwd_fact(q, k, v, 2, True)
    o1, _ = oracle.fwd_fact(3.5 * q + 0.25, 0.125 * k - 7.0, v, 2, True)
    np.testing.assert_allclose(o0, o1, rtol=1e-11, atol=1e-11)


@pytest.mark.parametrize("causal", [False, True])
def test_p1_closed_form(causal):
    """p = 1 (Sec. 2.2 with the quadratic term dropped, as Sec. 2.2 notes):
    o_i = (sum_n v_n + (sum_n v_n k^_n^T) q^_i) / (n_i + q^_i . sum_n k^_n)."""
    q, k, v = _rand(1, 1, 25, 6, 18)
    qh = (q - q.mean(-1, keepdims=True))
    qh /= np.sqrt((qh ** 2).mean(-1, keepdims=True))
    kh = (k - k.mean(-1, keepdims=True))
    kh /= np.sqrt((kh ** 2).mean(-1, keepdims=True))
    qh, kh, vv = qh[0, 0], kh[0, 0], v[0, 0]
    N = 25
    exp = np.empty((N, 6))
    for i in range(N):
        n = i + 1 if causal else N
        num = vv[:n].sum(0) + (vv[:n].T @ kh[:n]) @ qh[i]
        den = n + qh[i] @ kh[:n].sum(0)
        exp[i] = num / den
    o, _ = oracle.fwd_brute(q, k, v, 1, causal)
    np.testing.assert_allclose(o[0, 0], exp, rtol=1e-9, atol=1e-9)


def test_rows_sampler_matches_full():
    q, k, v = _rand(2, 3, 50, 8, 19)
    rows = np.array([0, 7, 49, 50, 123, 299])
    for causal in (False, True):
        o, g = oracle.fwd_brute(q, k, v, 2, causal)
        orow, grow = oracle.fwd_rows(q, k, v, 2, causal, rows)
        np.testing.assert_allclose(orow, o.reshape(-1, 8)[rows], rtol=1e-13)
        np.testing.assert_allclose(grow, g.reshape(-1)[rows], rtol=1e-13)


def test_bwd_finite_differences():
    check_bwd_finite_differences()


@pytest.mark.parametrize("p", [1, 2])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("D", [8, 64])
def test_bwd_torch_autograd(p, causal, D):
    torch = pytest.importorskip("torch")
    q, k, v = _rand(1, 2, 16, D, 20 + D)
    do = np.random.default_rng(5).standard_normal(q.shape)
    tq, tk, tv = (torch.tensor(a, dtype=torch.float64, requires_grad=True) for a in (q, k, v))

    def std(x):
        c = x - x.mean(-1, keepdim=True)
        return c / c.pow(2).mean(-1, keepdim=True).sqrt()

    s = std(tq) @ std(tk).transpose(-1, -2)
    w = sum(s ** l / math.factorial(l) for l in range(p + 1))
    if causal:
        w = w * torch.tril(torch.ones(16, 16, dtype=torch.float64))
    o = (w @ tv) / w.sum(-1, keepdim=True)
    (o * torch.tensor(do)).sum().backward()
    dq, dk, dv = oracle.bwd_brute(q, k, v, do, p, causal)
    for a, b in ((dq, tq.grad), (dk, tk.grad), (dv, tv.grad)):
        b = b.numpy()
        assert np.abs(a - b).max() <= 1e-9 * max(1.0, np.abs(b).max())


@pytest.mark.parametrize("causal", [False, True])
def test_bwd_invariants(causal):
    q, k, v = _rand(1, 1, 24, 16, 21)
    do = np.random.default_rng(6).standard_normal(q.shape)
    dq, dk, dv = oracle.bwd_brute(q, k, v, do, 2, causal)
    qh, _, _ = oracle.standardize(q)
    kh, _, _ = oracle.standardize(k)
    # shift invariance: sum_m dq_m = 0; scale invariance: dq . (q - mean) = 0
    np.testing.assert_allclose(dq.sum(-1), 0, atol=1e-10)
    np.testing.assert_allclose((dq * qh).sum(-1), 0, atol=1e-10)
    np.testing.assert_allclose(dk.sum(-1), 0, atol=1e-10)
    np.testing.assert_allclose((dk * kh).sum(-1), 0, atol=1e-10)
    # rows of A sum to one: sum_n dv_n = sum_i dO_i
    np.testing.assert_allclose(dv.sum(2), do.sum(2), atol=1e-10)


# --------------------------------------------------------------------------
# Planted mistakes: each must be caught by at least one pin above.
# --------------------------------------------------------------------------
MUTATIONS = {
    "drop_factorial": ("term *= s / (double)l;", "term *= s;"),
    "sample_std": ("var /= (double)D;                 /* population variance */",
                   "var /= (double)(D - 1);"),
    "exclusive_causal": ("long nend = causal ? i + 1 : N;\n    double g = 0.0, gabs",
                         "long nend = causal ? i : N;\n    double g = 0.0, gabs"),
    "fact_drop_half_g": ("g += 0.5 * tau * tau * quad;", "g += tau * tau * quad;"),
    "scale_brute_dropped": ("double w = f_taylor(tau * s, p);\n        g += w;",
                            "double w = f_taylor(s, p);\n        g += w;"),
    "scale_fact_quad_once": ("f += 0.5 * tau * tau * quad;", "f += 0.5 * tau * quad;"),
    "scale_fact_lin_g": ("double g = M->y1 + tau * lin;", "double g = M->y1 + lin;"),
    "scale_bwd_chain": ("double a = f_taylor(tau * s, p) / G[i];\n                double coef = tau * df_taylor",
                        "double a = f_taylor(tau * s, p) / G[i];\n                double coef = df_taylor"),
    "fact_transposed_x2": ("M->x2[j * D + m] += k[m] * vj;", "M->x2[m * D + j] += k[m] * vj;"),
    "fact_wrong_query_index": ("for (long l = 0; l < D; ++l) inner += q[l] * x3jm[l];",
                               "for (long l = 0; l < D; ++l) inner += q[m] * x3jm[l];"),
    "bwd_sign_dq": ("for (long d = 0; d < D; ++d) acc[d] += ds * kh[l * D + d];",
                    "for (long d = 0; d < D; ++d) acc[d] -= ds * kh[l * D + d];"),
    "bwd_std_sign": ("dx[d] = (dxh[d] - m1 - xh[d] * m2) / sig;",
                     "dx[d] = (dxh[d] - m1 + xh[d] * m2) / sig;"),
    "bwd_dv_index": ("accv[d] += a * dob[i * D + d];", "accv[d] += a * dob[l * D + d];"),
}

ALL_CHECKS = (check_golden_standardize, check_golden_forward, check_golden_backward,
              check_brute_vs_fact, check_bwd_finite_differences, check_scale_p1_closed_form,
              check_scale_p2_explicit, check_scale_small_limit,
              check_scale_bwd_finite_differences)


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
@pytest.mark.parametrize("mutation", sorted(MUTATIONS))
def test_planted_mistake_is_caught(mutation, tmp_path):
    src = open(os.path.join(os.path.dirname(oracle.__file__), "fastmax_ref.c")).read()
    old, new = MUTATIONS[mutation]
    assert src.count(old) == 1, mutation
    path_c = tmp_path / "mut.c"
    path_c.write_text(src.replace(old, new))
    path_so = tmp_path / "libmut.so"
    subprocess.run(["gcc", "-O1", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-o",
                    str(path_so), str(path_c), "-lm"], check=True)
    saved = oracle._lib
    oracle._lib = oracle._bind(str(path_so))
    caught = []
    try:
        for chk in ALL_CHECKS:
            try:
                with np.errstate(all="ignore"):
                    chk()
            except AssertionError:
                caught.append(chk.__name__)
    finally:
        oracle._lib = saved
    assert caught, f"planted mistake {mutation} went unnoticed"


def test_bwd_o_used_matches_exact_when_given_exact():
    q, k, v = _rand(1, 2, 20, 8, 22)
    do = np.random.default_rng(8).standard_normal(q.shape)
    for p in (1, 2):
        o, _ = oracle.fwd_brute(q, k, v, p, True)
        a = oracle.bwd_brute(q, k, v, do, p, True)
        b = oracle.bwd_brute(q, k, v, do, p, True, o_used=o)
        for x, y in zip(a, b):
            np.testing.assert_allclose(x, y, rtol=1e-12, atol=1e-12)
        # perturbing O moves only the c_i = dO.O/G terms: dv is unchanged
        c = oracle.bwd_brute(q, k, v, do, p, True, o_used=o * (1 + 1e-3))
        np.testing.assert_array_equal(c[2], a[2])
        assert np.abs(c[0] - a[0]).max() > 0

"""Pins for the oracle's quadratic-term dropout (CPU only).

The dropout of Sec. 2.4 (its dropout paragraph; "quadratic" in Fig. 2) masks
the D(D+1)/2 quadratic features k^_m k^_l (m <= l) of every key token, kept
ones scaled by 1/(1 - rate).  The checks tie the oracle to: the published
known-answer vectors of Philox4x32-10 (tests/golden), the unmasked oracle
(rate 0 with every bit kept is f_2), a closed form for one dropped feature
(which also fixes the feature numbering), the two independent formulations
(explicit weights and masked moments), the expectation over masks (inverted
dropout leaves E[F] and E[G] unchanged), central finite differences of the
backward, and the keep-bit layout re-derived from the generator.  Planted
mistakes in copies of the oracle source must each be caught.
"""
import json
import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand(B, H, N, D, seed):
    rng = np.random.default_rng([2402, 7901, 3000 + seed])
    return (rng.standard_normal((B, H, N, D)), rng.standard_normal((B, H, N, D)),
            rng.standard_normal((B, H, N, D)))


def _std(x):
    """Eqs. (6)-(7) written out: (x - mean) / population std over channels."""
    c = x - x.mean(-1, keepdims=True)
    return c / np.sqrt((c * c).mean(-1, keepdims=True))


def _pair(D, m, l):
    return m * D - m * (m - 1) // 2 + (l - m)


def _all_kept(B, H, N, D):
    nw = oracle.mask_words(D)
    bits = np.zeros((B, H, N, nw), dtype=np.uint32)
    npair = D * (D + 1) // 2
    for t in range(npair):
        bits[..., t // 32] |= np.uint32(1 << (t % 32))
    return bits


def _random_bits(B, H, N, D, keep, seed):
    rng = np.random.default_rng(seed)
    npair = D * (D + 1) // 2
    kept = rng.random((B, H, N, npair)) < keep
    nw = oracle.mask_words(D)
    bits = np.zeros((B, H, N, nw), dtype=np.uint32)
    for t in range(npair):
        bits[..., t // 32] |= kept[..., t].astype(np.uint32) << np.uint32(t % 32)
    return bits


# --------------------------------------------------------------------------
# checks (raise AssertionError); shared with the planted-mistake test
# --------------------------------------------------------------------------
def check_philox_kat():
    with open(os.path.join(GOLDEN, "philox4x32_10_kat.json")) as f:
        kat = json.load(f)
    for vec in kat["vectors"]:
        ctr = [int(x, 16) for x in vec["counter"]]
        key = [int(x, 16) for x in vec["key"]]
        out = [int(x, 16) for x in vec["out"]]
        got = [int(x) for x in oracle.philox4x32_10(ctr, key)]
        assert got == out, (vec, [hex(x) for x in got])


def check_rate0_all_kept_is_f2():
    q, k, v = _rand(1, 2, 23, 8, 1)
    do = np.random.default_rng(5).standard_normal(q.shape)
    bits = _all_kept(1, 2, 23, 8)
    for causal in (False, True):
        for tau in (1.0, 0.3):
            ref_o, ref_g = oracle.fwd_brute(q, k, v, 2, causal, scale=tau)
            for fn in (oracle.fwd_drop_brute, oracle.fwd_drop_fact):
                o, g = fn(q, k, v, bits, 0.0, causal, scale=tau)
                np.testing.assert_allclose(o, ref_o, rtol=1e-11, atol=1e-11)
                np.testing.assert_allclose(g, ref_g, rtol=1e-11)
            ref = oracle.bwd_brute(q, k, v, do, 2, causal, scale=tau)
            got = oracle.bwd_drop_brute(q, k, v, do, bits, 0.0, causal, scale=tau)
            for a, b in zip(got, ref):
                np.testing.assert_allclose(a, b, rtol=1e-9, atol=1e-10)


def check_single_dropped_feature():
    """N = 1: G = w_00.  Clearing feature t(m, l) at rate 0 lowers G by exactly
    c_ml tau^2 q^_m q^_l k^_m k^_l (c_mm = 1/2, c_ml = 1); at rate r with every
    bit kept the quadratic part of G is scaled by 1/(1 - r)."""
    D, tau = 6, 0.7
    q, k, v = _rand(1, 1, 1, D, 2)
    qh, kh = _std(q[0, 0, 0]) * tau, _std(k[0, 0, 0])
    full = _all_kept(1, 1, 1, D)
    _, g_full = oracle.fwd_drop_brute(q, k, v, full, 0.0, False, scale=tau)
    s = float(qh @ kh)
    quad = 0.5 * s * s
    np.testing.assert_allclose(g_full[0, 0, 0], 1 + s + quad, rtol=1e-12)
    for m, l in ((0, 0), (0, 3), (2, 5), (4, 4), (5, 5)):
        t = _pair(D, m, l)
        bits = full.copy()
        bits[..., t // 32] &= np.uint32(~(1 << (t % 32)) & 0xFFFFFFFF)
        for fn in (oracle.fwd_drop_brute, oracle.fwd_drop_fact):
            _, g = fn(q, k, v, bits, 0.0, False, scale=tau)
            c = 0.5 if m == l else 1.0
            want = c * qh[m] * qh[l] * kh[m] * kh[l]
            np.testing.assert_allclose(g_full[0, 0, 0] - g[0, 0, 0], want, rtol=1e-9,
                                       atol=1e-13)
    for r in (0.25, 0.5):
        for fn in (oracle.fwd_drop_brute, oracle.fwd_drop_fact):
            _, g = fn(q, k, v, full, r, False, scale=tau)
            np.testing.assert_allclose(g[0, 0, 0], 1 + s + quad / (1 - r), rtol=1e-12)


def check_drop_brute_vs_fact():
    for (B, H, N, D), causal, tau, r in (((1, 2, 31, 4), True, 1.0, 0.3),
                                         ((2, 1, 40, 8), False, 0.5, 0.6),
                                         ((1, 1, 35, 16), True, 0.25, 0.1)):
        q, k, v = _rand(B, H, N, D, N)
        bits = _random_bits(B, H, N, D, 1 - r, N)
        ob, gb = oracle.fwd_drop_brute(q, k, v, bits, r, causal, scale=tau)
        of, gf = oracle.fwd_drop_fact(q, k, v, bits, r, causal, scale=tau)
        np.testing.assert_allclose(of, ob, rtol=1e-9, atol=1e-10)
        np.testing.assert_allclose(gf, gb, rtol=1e-10)


def check_expectation_over_masks():
    """Inverted dropout: over masks with keep probability 1 - r the mean of the
    unnormalised F = O G and of G is the unmasked F and G (within 5 standard
    errors of the sample mean)."""
    B, H, N, D, r, K = 1, 1, 6, 4, 0.4, 400
    q, k, v = _rand(B, H, N, D, 3)
    o0, g0 = oracle.fwd_brute(q, k, v, 2, True)
    f0 = o0 * g0[..., None]
    fs, gs = [], []
    for s in range(K):
        bits = _random_bits(B, H, N, D, 1 - r, 100 + s)
        o, g = oracle.fwd_drop_brute(q, k, v, bits, r, True)
        fs.append(o * g[..., None])
        gs.append(g)
    for samples, ref in ((np.array(fs), f0), (np.array(gs), g0)):
        mean = samples.mean(0)
        se = samples.std(0, ddof=1) / np.sqrt(K)
        assert np.all(np.abs(mean - ref) <= 5 * se + 1e-12), np.max(np.abs(mean - ref) / (se + 1e-30))
    # row 0 sees only key 0, so a mask changes it; the check is not vacuous
    assert np.array(gs).std(0).max() > 0.01


def check_drop_bwd_finite_differences():
    B, H, N, D, r, tau = 1, 1, 9, 4, 0.3, 0.8
    q, k, v = _rand(B, H, N, D, 4)
    do = np.random.default_rng(9).standard_normal(q.shape)
    bits = _random_bits(B, H, N, D, 1 - r, 7)
    for causal in (True, False):
        dq, dk, dv = oracle.bwd_drop_brute(q, k, v, do, bits, r, causal, scale=tau)

        def loss(qq, kk, vv):
            o, _ = oracle.fwd_drop_brute(qq, kk, vv, bits, r, causal, scale=tau)
            return float((o * do).sum())
        h = 1e-6
        for which, grad in ((0, dq), (1, dk), (2, dv)):
            for idx in ((0, 0, 0, 0), (0, 0, 3, 2), (0, 0, N - 1, 1), (0, 0, 5, 3)):
                args = [q.copy(), k.copy(), v.copy()]
                args[which][idx] += h
                lp = loss(*args)
                args[which][idx] -= 2 * h
                lm = loss(*args)
                fd = (lp - lm) / (2 * h)
                assert abs(fd - grad[idx]) <= 1e-6 * max(1.0, abs(fd)), (which, idx, fd,
                                                                         grad[idx])


def check_mask_layout():
    """The keep bits re-derived from the (KAT-pinned) generator: counter
    (n, t // 4, head, 0), key (seed low, seed high), word t % 4, dropped iff
    below floor(rate 2^32); padding bits are zero; rate 0 keeps everything."""
    B, H, N, D, r, seed = 2, 3, 50, 16, 0.3, 0x1234567890ABCDEF
    bits = oracle.dropout_mask(B, H, N, D, r, seed)
    npair = D * (D + 1) // 2
    thr = int(np.floor(r * 2.0 ** 32))
    key = [seed & 0xFFFFFFFF, seed >> 32]
    rng = np.random.default_rng(0)
    for _ in range(300):
        b, h, n, t = (int(rng.integers(0, x)) for x in (B, H, N, npair))
        o = oracle.philox4x32_10([n, t // 4, b * H + h, 0], key)
        want = int(o[t % 4]) >= thr
        got = bool((int(bits[b, h, n, t // 32]) >> (t % 32)) & 1)
        assert got == want, (b, h, n, t)
    pad = npair % 32
    if pad:
        assert np.all(bits[..., -1] >> np.uint32(pad) == 0)
    ones = oracle.dropout_mask(1, 1, 5, D, 0.0, 7)
    np.testing.assert_array_equal(ones, _all_kept(1, 1, 5, D))
    kept = sum(bin(int(x)).count("1") for x in bits.reshape(-1))
    total = B * H * N * npair
    sd = np.sqrt(total * r * (1 - r))
    assert abs(kept - total * (1 - r)) <= 5 * sd, (kept, total)


def check_all_quadratic_dropped_is_p1():
    """With every quadratic feature dropped the masked weight is the p = 1
    weight 1 + tau s at any rate (the constant and linear terms are never
    dropped): the whole forward equals the unmasked p = 1 oracle, and a row
    with one key and tau s < -1 gets a negative G."""
    q, k, v = _rand(1, 2, 19, 8, 6)
    zero = np.zeros((1, 2, 19, oracle.mask_words(8)), dtype=np.uint32)
    for causal in (False, True):
        ref_o, ref_g = oracle.fwd_brute(q, k, v, 1, causal, scale=0.6)
        for fn in (oracle.fwd_drop_brute, oracle.fwd_drop_fact):
            o, g = fn(q, k, v, zero, 0.7, causal, scale=0.6)
            np.testing.assert_allclose(g, ref_g, rtol=1e-9, atol=1e-12)
            np.testing.assert_allclose(o * g[..., None], ref_o * ref_g[..., None],
                                       rtol=1e-9, atol=1e-9)
    qh, kh = _std(q[0, 0, 0]), _std(k[0, 0, 0])
    s = float(qh @ kh)
    kk = k[:, :, :1].copy()
    if s > -2:   # make tau s < -1 with tau = 1: k = -q gives s = -D
        kk = -q[:, :, :1].copy()
        s = -8.0
    _, g = oracle.fwd_drop_brute(q[:, :, :1], kk, v[:, :, :1], zero[:, :, :1], 0.5, False)
    np.testing.assert_allclose(g[0, 0, 0], 1 + s, rtol=1e-12)
    assert g[0, 0, 0] < 0


CHECKS = (check_philox_kat, check_rate0_all_kept_is_f2, check_single_dropped_feature,
          check_all_quadratic_dropped_is_p1,
          check_drop_brute_vs_fact, check_expectation_over_masks,
          check_drop_bwd_finite_differences, check_mask_layout)


@pytest.mark.parametrize("check", CHECKS, ids=lambda c: c.__name__)
def test_dropout_pin(check):
    check()


def test_masks_differ_across_tokens_heads_seeds():
    a = oracle.dropout_mask(1, 2, 8, 8, 0.5, 1)
    b = oracle.dropout_mask(1, 2, 8, 8, 0.5, 2)
    assert not np.array_equal(a, b)
    assert not np.array_equal(a[0, 0], a[0, 1])
    assert len({a[0, 0, n].tobytes() for n in range(8)}) == 8


# --------------------------------------------------------------------------
# Planted mistakes in the dropout code: each must be caught by a check above.
# --------------------------------------------------------------------------
MUTATIONS = {
    "philox_weyl": ("k1 += 0xBB67AE85u;", "k1 += 0xBB67AE84u;"),
    "philox_word_order": ("uint32_t n1 = (uint32_t)p1;", "uint32_t n1 = (uint32_t)p0;"),
    "mask_counter": ("(uint32_t)(t / 4), (uint32_t)hd, 0u}", "(uint32_t)(t % 4), (uint32_t)hd, 0u}"),
    "mask_bit_order": ("row[t / 32] |= 1u << (t % 32);", "row[t / 32] |= 1u << (31 - t % 32);"),
    "pair_numbering": ("return m * D - m * (m - 1) / 2 + (l - m);",
                       "return l * (l + 1) / 2 + m;"),
    "weight_diag_half": ("double c = (l == m) ? 0.5 : 1.0;\n            quad += c",
                         "double c = 1.0;\n            quad += c"),
    "dropped_not_zero": ("? inv_keep : 0.0;", "? inv_keep : 1.0;"),
    "no_inverted_scale": ("double inv_keep = 1.0 / (1.0 - rate);\n    for (long hd = 0; hd < heads; ++hd) {\n        double *qh",
                          "double inv_keep = 1.0;\n    for (long hd = 0; hd < heads; ++hd) {\n        double *qh"),
    "fact_masks_linear": ("X2[m * D1 + j] += kn[m] * vp[j];",
                          "X2[m * D1 + j] += kn[m] * vp[j] * keep_mult(row, m, inv_keep);"),
    "fact_exclusive_causal": ("if (causal) DROP_ADD(i);\n            const double *qi",
                              "const double *qi"),
    "bwd_h_unmasked": ("acc += qi[l] * kn[l] * keep_mult(row, t, inv_keep);\n                    }\n                    h[a] = acc;\n                }\n                for (long a = 0; a < D; ++a) dqt",
                       "acc += qi[l] * kn[l];\n                    }\n                    h[a] = acc;\n                }\n                for (long a = 0; a < D; ++a) dqt"),
    "bwd_dk_h_missing": ("dkh[n * D + a] += dw * qi[a] * h[a];", "dkh[n * D + a] += dw * qi[a];"),
    "bwd_dv_unnormalised": ("dvh[n * D + a] += w * dob[i * D + a] / G[i];",
                            "dvh[n * D + a] += w * dob[i * D + a];"),
    "bwd_tau_chain": ("for (long a = 0; a < D; ++a) dqh[a] = tau * dqt[r * D + a];",
                      "for (long a = 0; a < D; ++a) dqh[a] = dqt[r * D + a];"),
}


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
@pytest.mark.parametrize("mutation", sorted(MUTATIONS))
def test_planted_dropout_mistake_is_caught(mutation, tmp_path):
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
        for chk in CHECKS:
            try:
                with np.errstate(all="ignore"):
                    chk()
            except AssertionError:
                caught.append(chk.__name__)
    finally:
        oracle._lib = saved
    assert caught, f"planted mistake {mutation} went unnoticed"

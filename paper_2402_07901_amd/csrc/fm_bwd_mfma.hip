// Causal Fastmax backward on CDNA4 MFMA, head dimension 64, p = 2, bf16 I/O.
//
// The custom gradient of Sec. 2.5: only G is kept from the forward, q^ and
// k^ are recomputed, and every N x N quantity is replaced by moments.  With
// u_i = dO_i / G_i, c_i = (dO_i . O_i) / G_i, u~_i = [u_i, -c_i], v'_n = [v_n, 1]
// and the score derivative of Sec. 2.3 (Eq. "bound": d a_in / d s_il =
// f'(s_il) / G_i (delta_nl - a_in), f_2' = 1 + s):
//
//   dq^_i = sum_{n<=i} (1 + s_in)(u~_i . v'_n) k^_n
//   dk^_n = sum_{i>=n} (1 + s_in)(u~_i . v'_n) q^_i
//   dv_n  = sum_{i>=n} f(s_in) u_i
//
// Kernels:
//  bwd_prep     1/G, c per token; per head max|u|, max|v|, max|c| (fp16 scales).
//  (dv)         the causal scan run in reverse with values u (no divide),
//               launched together with bwd_intra.
//  bwd_intra    in-chunk pairs (both n <= i inside a 128-token chunk) of dq^ and
//               dk^ on MFMA; initialises the fp32 accumulators dq^, dk^.
//  bwd_mg_scan  the inter-chunk part, one kernel for both gradients:
//                 out_t[l] = sum_s (1 + x^_t . y^_s)(z_t . w_s) y^_s[l]
//               over the summed tokens s of earlier chunks in scan order,
//               factorised (p = 1 in the weights, times a rank-(D+1) term):
//                 out_t[l] = sum_{m,j} x^_tm z_tj X3[m][l][j] + sum_j z_tj M1[j][l]
//               with X3[m][l][j] = sum_s y^_sm y^_sl w_sj and M1 = sum_s w_sj y^_sl
//               (j over the D+1 columns).  dq^: x = q, y = k, z = u~, w = v',
//               chunks in order.  dk^: x = k, y = q, z = v', w = u~, chunks in
//               reverse order (X3 is then the T3 moment, M1 the T2 moment).
//  bwd_finish   back through the standardisation (Eqs. 6-7).
#include <hip/hip_runtime.h>

#include <limits.h>

#include "fm_causal_scan.h"
#include "fm_common.h"
#include "fm_internal.h"
#include "fm_mfma.h"

namespace fm {
namespace mfma_bwd {

using namespace mx;

constexpr int C = 128;   // tokens per chunk

// ---------------------------------------------------------------------------
// bwd_prep: one workgroup per (head, 128-token chunk), an octet of lanes per
// token; per-chunk maxima go to pmax[head][chunk][4].  Also standardises q and
// k once for the whole backward (Sec. 2.2, Eqs. 6-7): q^, k^ in fp16, which
// the scans read instead of recomputing them (bwd_finish, which needs them in
// fp32 for the cancellation-prone standardisation backward, recomputes them).

__global__ __launch_bounds__(256) void bwd_prep(const bf16_t *__restrict__ q,
                                                const bf16_t *__restrict__ k,
                                                const bf16_t *__restrict__ o,
                                                const bf16_t *__restrict__ dout,
                                                const bf16_t *__restrict__ v,
                                                const float *__restrict__ g,
                                                float *__restrict__ rg, float *__restrict__ cc,
                                                float *__restrict__ pmax, _Float16 *__restrict__ qh,
                                                _Float16 *__restrict__ kh, int N, int nch, float qs,
                                                unsigned int *__restrict__ flags, int nflags)
{
    __shared__ float red[3][4];
    // the segment flags of the dv scan that follows start lowered
    if (blockIdx.x == 0)
        for (int i = threadIdx.x; i < nflags; i += 256) flags[i] = 0u;
    const int head = blockIdx.x / nch, c = blockIdx.x % nch, tid = threadIdx.x;
    const size_t hb = (size_t)head * N;
    q += hb * D;
    k += hb * D;
    qh += hb * D;
    kh += hb * D;
    o += hb * D;
    dout += hb * D;
    v += hb * D;
    g += hb;
    rg += hb;
    cc += hb;
    const int oc = tid >> 3, cg = tid & 7;
    float umax = 0.f, vmax = 0.f, cmax = 0.f;
    for (int n0 = c * C; n0 < min(N, (c + 1) * C); n0 += 32) {
        const int n = n0 + oc;
        const bool valid = n < N;
        float xo[8] = {}, xd[8] = {}, xv[8] = {};
        float r = 0.f;
        if (valid) {
            bf16x8_to_f32(*(const uint4 *)(o + (size_t)n * D + 8 * cg), xo);
            bf16x8_to_f32(*(const uint4 *)(dout + (size_t)n * D + 8 * cg), xd);
            bf16x8_to_f32(*(const uint4 *)(v + (size_t)n * D + 8 * cg), xv);
            r = 1.0f / g[n];
        }
        float dot = 0.f, am = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            dot = fmaf(xd[i], xo[i], dot);
            am = fmaxf(am, fabsf(xd[i]));
            vmax = fmaxf(vmax, fabsf(xv[i]));
        }
        dot = octet_sum(dot);
        const float c = dot * r;
        umax = fmaxf(umax, am * fabsf(r));
        cmax = fmaxf(cmax, fabsf(c));
        if (valid && cg == 0) {
            rg[n] = r;
            cc[n] = c;
        }
        if (valid) {
            float x[8];
            bf16x8_to_f32(*(const uint4 *)(q + (size_t)n * D + 8 * cg), x);
            *(h8 *)(qh + (size_t)n * D + 8 * cg) = standardise8(x, true, qs);
            bf16x8_to_f32(*(const uint4 *)(k + (size_t)n * D + 8 * cg), x);
            *(h8 *)(kh + (size_t)n * D + 8 * cg) = standardise8(x, true);
        }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        umax = fmaxf(umax, __shfl_xor(umax, off));
        vmax = fmaxf(vmax, __shfl_xor(vmax, off));
        cmax = fmaxf(cmax, __shfl_xor(cmax, off));
    }
    if ((tid & 63) == 0) {
        red[0][tid >> 6] = umax;
        red[1][tid >> 6] = vmax;
        red[2][tid >> 6] = cmax;
    }
    __syncthreads();
    if (tid < 3) {
        float m = 0.f;
        for (int w = 0; w < 4; ++w) m = fmaxf(m, red[tid][w]);
        pmax[((size_t)head * nch + c) * 4 + tid] = m;
    }
}

// per-head maxima over the chunks: [0] max|u|, [1] max|v|, [2] max|c|
struct HeadMax {
    float u, v, c;
};
__device__ __forceinline__ HeadMax head_max(const float *pmax, int head, int nch)
{
    HeadMax r{0.f, 0.f, 0.f};
    const float *p = pmax + (size_t)head * nch * 4;
    // unrolled so that several scalar loads are in flight per wait
#pragma unroll 8
    for (int c = 0; c < nch; ++c) {
        r.u = fmaxf(r.u, p[4 * c]);
        r.v = fmaxf(r.v, p[4 * c + 1]);
        r.c = fmaxf(r.c, p[4 * c + 2]);
    }
    return r;
}

// ---------------------------------------------------------------------------
// bwd_intra: (head, chunk); eight waves: 0-3 the dq^ row tiles, 4-7 the dk^
// key tiles, two each ({v, 7-v}: 9 of the chunk's 36 tile pairs per wave).

struct ISmem {
    _Float16 qrow[C * RS64];   // q^ [t][m]
    _Float16 krow[C * RS64];   // k^ [s][m]
    _Float16 vrow[C * RS64];   // v * 2^-ev [s][j]
    _Float16 urow[C * RS64];   // u * 2^-eu [t][j]
    _Float16 qT[D * RS128];    // q^ [m][t]
    _Float16 kT[D * RS128];    // k^ [m][s]
    float cc[C];
};

__device__ __forceinline__ void intra_block(ISmem &sm, const _Float16 *__restrict__ q,
                                            const _Float16 *__restrict__ k,
                                            const bf16_t *__restrict__ v,
                                            const bf16_t *__restrict__ dout,
                                            const float *__restrict__ rg,
                                            const float *__restrict__ cc,
                                            const float *__restrict__ hmax,
                                            float *__restrict__ dqh, float *__restrict__ dkh, int N,
                                            int nch, int blk)
{
    const int head = blk / nch, c = blk % nch;
    const int n0 = c * C;
    const size_t hb = (size_t)head * N;
    q += hb * D;
    k += hb * D;
    v += hb * D;
    dout += hb * D;
    rg += hb;
    cc += hb;
    dqh += hb * D;
    dkh += hb * D;

    const HeadMax hm = head_max(hmax, head, nch);
    const int ev = pow2_exponent(hm.v), eu = pow2_exponent(hm.u);
    // |P| <= 65 (64 max|v| max|u| + max|c|)
    const int ep = pow2_exponent(65.0f * fmaf(64.0f * hm.v, hm.u, hm.c));
    const float sv = ldexpf(1.0f, -ev), su = ldexpf(1.0f, -eu);
    const float sa = ldexpf(1.0f, ev + eu), sp = ldexpf(1.0f, -ep), so = ldexpf(1.0f, ep);

    const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, r16 = lane & 15, h = lane >> 4;
    // staging: four passes of 32 tokens, an octet of lanes per token
    {
        const int oc = tid >> 3, cg = tid & 7;
        for (int pass = 0; pass < 2; ++pass) {
            const int t = 64 * pass + oc, n = n0 + t;
            const bool valid = n < N;
            float xv[8] = {}, xu[8] = {};
            h8 hq = {0, 0, 0, 0, 0, 0, 0, 0}, hk = hq;
            float r = 0.f;
            if (valid) {
                hq = *(const h8 *)(q + (size_t)n * D + 8 * cg);
                hk = *(const h8 *)(k + (size_t)n * D + 8 * cg);
                bf16x8_to_f32(*(const uint4 *)(v + (size_t)n * D + 8 * cg), xv);
                bf16x8_to_f32(*(const uint4 *)(dout + (size_t)n * D + 8 * cg), xu);
                r = rg[n];
            }
            h8 hv, hu;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                hv[i] = (_Float16)(xv[i] * sv);
                hu[i] = (_Float16)(xu[i] * (r * su));
            }
            *(h8 *)(sm.qrow + sw64(t, 8 * cg)) = hq;
            *(h8 *)(sm.krow + sw64(t, 8 * cg)) = hk;
            *(h8 *)(sm.vrow + sw64(t, 8 * cg)) = hv;
            *(h8 *)(sm.urow + sw64(t, 8 * cg)) = hu;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                sm.qT[swx(8 * cg + i, t)] = hq[i];
                sm.kT[swx(8 * cg + i, t)] = hk[i];
            }
            if (cg == 0) sm.cc[t] = valid ? cc[n] : 0.f;
        }
    }
    __syncthreads();

    const h4 z4 = {0, 0, 0, 0};
    const int v4 = w & 3;
    // dq^ (waves 0-3): query tiles rt in {v4, 7-v4}; lane column t = 16 rt + r16
    if (w < 4)
    for (int pick = 0; pick < 2; ++pick) {
        const int rt = pick ? 7 - v4 : v4;
        const int t = 16 * rt + r16;
        const float ct = sm.cc[t];
        const h8 QB0 = ld8(sm.qrow + sw64(t, 8 * h)), QB1 = ld8(sm.qrow + sw64(t, 32 + 8 * h));
        const h8 UB0 = ld8(sm.urow + sw64(t, 8 * h)), UB1 = ld8(sm.urow + sw64(t, 32 + 8 * h));
        // P[s][t] of key tile st: lane (column t, rows s = 16 st + 4h + i)
        auto ptile = [&](int st) -> h4 {
            f4 S = {0.f, 0.f, 0.f, 0.f}, A = {0.f, 0.f, 0.f, 0.f};
            S = mfma(ld8(sm.krow + sw64(16 * st + r16, 8 * h)), QB0, S);
            S = mfma(ld8(sm.krow + sw64(16 * st + r16, 32 + 8 * h)), QB1, S);
            A = mfma(ld8(sm.vrow + sw64(16 * st + r16, 8 * h)), UB0, A);
            A = mfma(ld8(sm.vrow + sw64(16 * st + r16, 32 + 8 * h)), UB1, A);
            f4 P;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                float pv = (1.0f + S[i]) * fmaf(A[i], sa, -ct) * sp;
                if (st == rt && 4 * h + i > r16) pv = 0.f;
                P[i] = pv;
            }
            return cvt4(P);
        };
        f4 acc[4];
#pragma unroll
        for (int lt = 0; lt < 4; ++lt) acc[lt] = f4{0.f, 0.f, 0.f, 0.f};
        for (int a = 0; a <= rt; a += 2) {
            const int b = a + 1;
            const h4 pa = ptile(a);
            const h4 pb = b <= rt ? ptile(b) : z4;
            const h8 B = cat(pa, pb);
#pragma unroll
            for (int lt = 0; lt < 4; ++lt) {
                const h4 ka = ld4(sm.kT + swx(16 * lt + r16, 16 * a + 4 * h));
                const h4 kb = b <= rt ? ld4(sm.kT + swx(16 * lt + r16, 16 * b + 4 * h)) : z4;
                acc[lt] = mfma(cat(ka, kb), B, acc[lt]);
            }
        }
        if (n0 + t < N) {
#pragma unroll
            for (int lt = 0; lt < 4; ++lt)
                *(f4 *)(dqh + (size_t)(n0 + t) * D + 16 * lt + 4 * h) = acc[lt] * so;
        }
    }
    // dk^ (waves 4-7): key tiles rs in {v4, 7-v4}; lane column s = 16 rs + r16
    if (w >= 4)
    for (int pick = 0; pick < 2; ++pick) {
        const int rs = pick ? 7 - v4 : v4;
        const int s = 16 * rs + r16;
        const h8 KB0 = ld8(sm.krow + sw64(s, 8 * h)), KB1 = ld8(sm.krow + sw64(s, 32 + 8 * h));
        const h8 VB0 = ld8(sm.vrow + sw64(s, 8 * h)), VB1 = ld8(sm.vrow + sw64(s, 32 + 8 * h));
        // P^T[t][s] of query tile tt: lane (column s, rows t = 16 tt + 4h + i)
        auto pttile = [&](int tt) -> h4 {
            f4 S = {0.f, 0.f, 0.f, 0.f}, A = {0.f, 0.f, 0.f, 0.f};
            S = mfma(ld8(sm.qrow + sw64(16 * tt + r16, 8 * h)), KB0, S);
            S = mfma(ld8(sm.qrow + sw64(16 * tt + r16, 32 + 8 * h)), KB1, S);
            A = mfma(ld8(sm.urow + sw64(16 * tt + r16, 8 * h)), VB0, A);
            A = mfma(ld8(sm.urow + sw64(16 * tt + r16, 32 + 8 * h)), VB1, A);
            f4 P;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float ct = sm.cc[16 * tt + 4 * h + i];
                float pv = (1.0f + S[i]) * fmaf(A[i], sa, -ct) * sp;
                if (tt == rs && 4 * h + i < r16) pv = 0.f;
                P[i] = pv;
            }
            return cvt4(P);
        };
        f4 acc[4];
#pragma unroll
        for (int lt = 0; lt < 4; ++lt) acc[lt] = f4{0.f, 0.f, 0.f, 0.f};
        for (int a = rs; a < 8; a += 2) {
            const int b = a + 1;
            const h4 pa = pttile(a);
            const h4 pb = b < 8 ? pttile(b) : z4;
            const h8 B = cat(pa, pb);
#pragma unroll
            for (int lt = 0; lt < 4; ++lt) {
                const h4 qa = ld4(sm.qT + swx(16 * lt + r16, 16 * a + 4 * h));
                const h4 qb = b < 8 ? ld4(sm.qT + swx(16 * lt + r16, 16 * b + 4 * h)) : z4;
                acc[lt] = mfma(cat(qa, qb), B, acc[lt]);
            }
        }
        if (n0 + s < N) {
#pragma unroll
            for (int lt = 0; lt < 4; ++lt)
                *(f4 *)(dkh + (size_t)(n0 + s) * D + 16 * lt + 4 * h) = acc[lt] * so;
        }
    }
}

// ---------------------------------------------------------------------------
// bwd_mg_scan: (head, 16-column output tile L); eight waves, two per SIMD,
// each holding X3[m][l in L][j] for its 8 channels m = 8w.. as 32
// accumulator tiles (rows j, columns l) in registers.

constexpr int MG_NW = 8;
constexpr int MG_NTH = MG_NW * 64;
constexpr int MG_MPW = D / MG_NW;   // channels per wave

struct GSmem {
    _Float16 xrow[C * RS64];      // x^ [t][m] of the chunk being contracted
    _Float16 zrow[C * RS64];      // z * 2^-ez [t][j]
    _Float16 yT[D * RS128];       // y^ [m][s] of the chunk added to the moments
    _Float16 wT[D * RS128];       // w * 2^-ew [j][s]
    _Float16 wDh[C];              // w_D * 2^-eD [s]
    float zD[C];                  // z_D * 2^(eD - ew - ez) [t]
    float fpart[MG_NW * 4 * C * 4];   // [wave][row quad][t][4]
    float m1g[16];                // sum_s w_D y^_sl (units 2^-eD), l in L
    f4 ex[4][3][64];              // the extra accumulator tiles of waves 0-3, between uses
};

template <int DIR, bool CAUSAL>
__device__ __forceinline__ void mg_scan(GSmem &sm, int b, int nblk,
                                        const _Float16 *__restrict__ x,
                                        const _Float16 *__restrict__ y,
                                        const bf16_t *__restrict__ z,
                                        const bf16_t *__restrict__ wv,
                                        const float *__restrict__ rg,
                                        const float *__restrict__ cc,
                                        const float *__restrict__ hmax, float *__restrict__ dxh,
                                        int N, int BH)
{
    // the four output tiles of a head on one XCD (shared x, y, z, w rows in L2);
    // b counts from the first block of this scan, whose id is a multiple of 8
    int head, L;
    if ((nblk & 31) == 0) {
        const int xcd = b & 7, idx = b >> 3;
        L = idx & 3;
        head = (idx >> 2) * 8 + xcd;
    } else {
        head = b >> 2;
        L = b & 3;
    }
    if (head >= BH) return;
    const size_t hb = (size_t)head * N;
    x += hb * D;
    y += hb * D;
    z += hb * D;
    wv += hb * D;
    rg += hb;
    cc += hb;
    dxh += hb * D;

    // roles: DIR 0 (dq^): z = u (row scale 1/G), z_D = -c, w = v, w_D = 1;
    //        DIR 1 (dk^): z = v, z_D = 1, w = u, w_D = -c.
    const HeadMax hm = head_max(hmax, head, (N + C - 1) / C);
    const float zmax = DIR ? hm.v : hm.u, wmax = DIR ? hm.u : hm.v;
    const float wdmax = DIR ? hm.c : 1.0f;
    const int ew = pow2_exponent(64.0f * (float)N * wmax);
    const int ez = pow2_exponent(zmax);
    const int ed = pow2_exponent(64.0f * (float)N * wdmax);
    const float sw = ldexpf(1.0f, -ew), sz = ldexpf(1.0f, -ez), sd = ldexpf(1.0f, -ed);
    const float szd = ldexpf(1.0f, ed - ew - ez), sout = ldexpf(1.0f, ew + ez);

    int tid = threadIdx.x;
    const int w = tid >> 6;
    int lane = tid & 63, r16 = lane & 15, h = lane >> 4;
    auto refresh_ids = [&]() {
        asm volatile("" : "+v"(tid));
        lane = tid & 63;
        r16 = lane & 15;
        h = lane >> 4;
    };

    // X3 of the wave's channels in fp16, paired per contraction K step (j
    // tiles 2p, 2p+1); rebuilt in fp32 for each update (one MFMA per tile
    // against a 0/1 permutation matrix) and rounded back once per chunk
    h8 Ast[MG_MPW][2];
#pragma unroll
    for (int m = 0; m < MG_MPW; ++m) Ast[m][0] = Ast[m][1] = h8{0, 0, 0, 0, 0, 0, 0, 0};
    // extra tiles (waves 0-3): wave 0 M1 (j tiles 0,1) and M1G; wave 1 M1 (j
    // tiles 2,3); waves 2,3 X3G = sum_s w_D y^_sm y^_sl for m tiles 2(w-2),
    // 2(w-2)+1; kept in LDS between uses
    if (w < 4) {
#pragma unroll
        for (int e = 0; e < 3; ++e) sm.ex[w][e][lane] = f4{0.f, 0.f, 0.f, 0.f};
    }

    const int nch = (N + C - 1) / C;
    auto chunk_of = [&](int kk) { return DIR ? nch - 1 - kk : kk; };

    // staging of chunk c: lanes of an octet share a token; a thread takes
    // tokens 2tg, 2tg+1 (tg = tid/8), channels 8(tid%8)..
    uint4 px[2], py[2], pz[2], pw[2];
    float prg[2], pcc[2];
    auto prefetch = [&](int c) {
        const uint4 zero = {0u, 0u, 0u, 0u};
        const int tg = tid >> 3, cg = tid & 7;
#pragma unroll
        for (int e = 0; e < 2; ++e) {
            const int n = c * C + 2 * tg + e;
            px[e] = py[e] = pz[e] = pw[e] = zero;
            prg[e] = pcc[e] = 0.f;
            if (n < N) {
                px[e] = *(const uint4 *)(x + (size_t)n * D + 8 * cg);
                py[e] = *(const uint4 *)(y + (size_t)n * D + 8 * cg);
                pz[e] = *(const uint4 *)(z + (size_t)n * D + 8 * cg);
                pw[e] = *(const uint4 *)(wv + (size_t)n * D + 8 * cg);
                prg[e] = rg[n];
                pcc[e] = cc[n];
            }
        }
    };
    // the output side (x^ rows, scaled z rows, z_D)
    auto stage_xz = [&](int c) {
        const int tg = tid >> 3, cg = tid & 7;
#pragma unroll
        for (int e = 0; e < 2; ++e) {
            const int t = 2 * tg + e;
            const bool valid = c * C + t < N;
            float f[8];
            *(h8 *)(sm.xrow + sw64(t, 8 * cg)) = __builtin_bit_cast(h8, px[e]);
            const float zs = (DIR ? 1.0f : prg[e]) * sz;
            bf16x8_to_f32(pz[e], f);
            h8 hz;
#pragma unroll
            for (int i = 0; i < 8; ++i) hz[i] = (_Float16)(f[i] * zs);
            *(h8 *)(sm.zrow + sw64(t, 8 * cg)) = hz;
            if (cg == 0) sm.zD[t] = valid ? (DIR ? 1.0f : -pcc[e]) * szd : 0.f;
        }
    };
    // the summed side (y^ and scaled w transposed, w_D)
    auto stage_yw = [&](int c) {
        const int tg = tid >> 3, cg = tid & 7;
        h8 hy[2], hw[2];
#pragma unroll
        for (int e = 0; e < 2; ++e) {
            const int t = 2 * tg + e;
            const bool valid = c * C + t < N;
            float f[8];
            hy[e] = __builtin_bit_cast(h8, py[e]);
            const float ws = (DIR ? prg[e] : 1.0f) * sw;
            bf16x8_to_f32(pw[e], f);
#pragma unroll
            for (int i = 0; i < 8; ++i) hw[e][i] = (_Float16)(f[i] * ws);
            if (cg == 0) sm.wDh[t] = (_Float16)(valid ? (DIR ? -pcc[e] : 1.0f) * sd : 0.f);
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            *(h2 *)(sm.yT + swx(8 * cg + i, 2 * tg)) = h2{hy[0][i], hy[1][i]};
            *(h2 *)(sm.wT + swx(8 * cg + i, 2 * tg)) = h2{hw[0][i], hw[1][i]};
        }
    };

    // (A) contraction of the staged output side (chunk c) with the moments
    // accumulated so far; partial outputs to LDS
    auto contract = [&]() {
        if (w == 0 && h == 0) sm.m1g[r16] = sm.ex[0][2][lane][0];
        h8 Aex = {0, 0, 0, 0, 0, 0, 0, 0};
        if (w < 4) Aex = cat(cvt4(sm.ex[w][0][lane]), cvt4(sm.ex[w][1][lane]));
#pragma unroll 1
        for (int rt = 0; rt < C / 16; ++rt) {
            const int t = 16 * rt + r16;
            const h8 xv = ld8(sm.xrow + sw64(t, MG_MPW * w));
            h8 Zb[2];
#pragma unroll
            for (int p = 0; p < 2; ++p)
                Zb[p] = cat(ld4(sm.zrow + sw64(t, 32 * p + 4 * h)),
                            ld4(sm.zrow + sw64(t, 32 * p + 16 + 4 * h)));
            f4 Dout = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int mm = 0; mm < MG_MPW; ++mm) {
                f4 E = {0.f, 0.f, 0.f, 0.f};
                E = mfma(Ast[mm][0], Zb[0], E);
                E = mfma(Ast[mm][1], Zb[1], E);
                const float xm = (float)xv[mm];
#pragma unroll
                for (int i = 0; i < 4; ++i) Dout[i] = fmaf(xm, E[i], Dout[i]);
            }
            if (w < 4) {
                const float zd = sm.zD[t];
                if (w < 2) {
                    // z at this wave's M1 column pair
                    const h8 Zw = cat(ld4(sm.zrow + sw64(t, 32 * w + 4 * h)),
                                      ld4(sm.zrow + sw64(t, 32 * w + 16 + 4 * h)));
                    Dout = mfma(Aex, Zw, Dout);
                    if (w == 0) {
#pragma unroll
                        for (int i = 0; i < 4; ++i) Dout[i] = fmaf(zd, sm.m1g[4 * h + i], Dout[i]);
                    }
                } else {
                    const h8 Xb = cat(ld4(sm.xrow + sw64(t, 32 * (w - 2) + 4 * h)),
                                      ld4(sm.xrow + sw64(t, 32 * (w - 2) + 16 + 4 * h)));
                    f4 Eg = {0.f, 0.f, 0.f, 0.f};
                    Eg = mfma(Aex, Xb, Eg);
#pragma unroll
                    for (int i = 0; i < 4; ++i) Dout[i] = fmaf(zd, Eg[i], Dout[i]);
                }
            }
            *(f4 *)(sm.fpart + ((w * 4 + h) * C + t) * 4) = Dout;
        }
    };
    // the waves' partial outputs of chunk c summed into dx^ (added to the
    // in-chunk part when causal, stored when the moments are totals)
    auto combine = [&](int c) {
        const int t = tid & (C - 1), qd = tid >> 7;
        const int n = c * C + t;
        if (n < N) {
            f4 F = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ww = 0; ww < MG_NW; ++ww)
                F += *(const f4 *)(sm.fpart + ((ww * 4 + qd) * C + t) * 4);
            f4 *dst = (f4 *)(dxh + (size_t)n * D + 16 * L + 4 * qd);
            if constexpr (CAUSAL) *dst = *dst + F * sout;
            else *dst = F * sout;
        }
    };
    // (B) moments += the staged summed side (chunk c), 32 tokens per K step,
    // on fp32 tiles rebuilt from the fp16 pairs
    auto update = [&]() {
        h8 pa = {0, 0, 0, 0, 0, 0, 0, 0}, pb = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
            const bool on = h == (r16 >> 2) && jj == (r16 & 3);
            pa[jj] = on ? (_Float16)1.0f : (_Float16)0.0f;
            pb[4 + jj] = on ? (_Float16)1.0f : (_Float16)0.0f;
        }
        f4 acc[MG_MPW][4];
#pragma unroll
        for (int m = 0; m < MG_MPW; ++m)
#pragma unroll
            for (int jt = 0; jt < 4; ++jt)
                acc[m][jt] = mfma((jt & 1) ? pb : pa, Ast[m][jt >> 1], f4{0.f, 0.f, 0.f, 0.f});
#pragma unroll 1
        for (int ks = 0; ks < C / 32; ++ks) {
            const int col = 32 * ks + 8 * h;
            h8 Aw[4];
#pragma unroll
            for (int jt = 0; jt < 4; ++jt) Aw[jt] = ld8(sm.wT + swx(16 * jt + r16, col));
            const h8 Yl = ld8(sm.yT + swx(16 * L + r16, col));
#pragma unroll
            for (int m = 0; m < MG_MPW; ++m) {
                const h8 Ym = ld8(sm.yT + swx(MG_MPW * w + m, col));
                const h8 Bm = Ym * Yl;
#pragma unroll
                for (int jt = 0; jt < 4; ++jt) acc[m][jt] = mfma(Aw[jt], Bm, acc[m][jt]);
            }
            if (w < 4) {
                const h8 WD = ld8(sm.wDh + col);
                f4 ex[3];
#pragma unroll
                for (int e = 0; e < 3; ++e) ex[e] = sm.ex[w][e][lane];
                if (w == 0) {
                    ex[0] = mfma(Aw[0], Yl, ex[0]);
                    ex[1] = mfma(Aw[1], Yl, ex[1]);
                    const h8 zero8 = {0, 0, 0, 0, 0, 0, 0, 0};
                    ex[2] = mfma(r16 == 0 ? WD : zero8, Yl, ex[2]);
                } else if (w == 1) {
                    ex[0] = mfma(Aw[2], Yl, ex[0]);
                    ex[1] = mfma(Aw[3], Yl, ex[1]);
                } else {
                    const h8 YW = Yl * WD;
#pragma unroll
                    for (int e = 0; e < 2; ++e) {
                        const int mt = 2 * (w - 2) + e;
                        ex[e] = mfma(ld8(sm.yT + swx(16 * mt + r16, col)), YW, ex[e]);
                    }
                }
#pragma unroll
                for (int e = 0; e < 3; ++e) sm.ex[w][e][lane] = ex[e];
            }
        }
#pragma unroll
        for (int m = 0; m < MG_MPW; ++m)
#pragma unroll
            for (int p = 0; p < 2; ++p) Ast[m][p] = cat(cvt4(acc[m][2 * p]), cvt4(acc[m][2 * p + 1]));
    };

    if constexpr (CAUSAL) {
        prefetch(chunk_of(0));
        stage_xz(chunk_of(0));
        stage_yw(chunk_of(0));
        __syncthreads();
        for (int kk = 0; kk < nch; ++kk) {
            const int c = chunk_of(kk);
            const bool more = kk + 1 < nch;
            __builtin_amdgcn_sched_barrier(0);
            refresh_ids();
            // (A) chunk c against the moments of earlier chunks
            if (kk > 0) contract();
            __syncthreads();
            // (B) chunk c's contribution out, the moments updated with chunk
            //     c, the output side of the next chunk staged
            __builtin_amdgcn_sched_barrier(0);
            refresh_ids();
            if (kk > 0) combine(c);
            if (more) prefetch(chunk_of(kk + 1));
            update();
            if (more) stage_xz(chunk_of(kk + 1));
            __syncthreads();
            // (C) the summed side of the next chunk (after the update)
            if (more) {
                stage_yw(chunk_of(kk + 1));
                __syncthreads();
            }
        }
    } else {
        // totals (Sec. 2.5 with every pair (s, t) present): the moments of
        // all chunks first, then every chunk contracted against them
        prefetch(0);
        stage_yw(0);
        __syncthreads();
        for (int c = 0; c < nch; ++c) {
            const bool more = c + 1 < nch;
            __builtin_amdgcn_sched_barrier(0);
            refresh_ids();
            if (more) prefetch(c + 1);
            update();
            __syncthreads();
            if (more) {
                stage_yw(c + 1);
                __syncthreads();
            }
        }
        prefetch(0);
        stage_xz(0);
        __syncthreads();
        for (int c = 0; c < nch; ++c) {
            const bool more = c + 1 < nch;
            __builtin_amdgcn_sched_barrier(0);
            refresh_ids();
            contract();
            if (more) prefetch(c + 1);
            __syncthreads();
            __builtin_amdgcn_sched_barrier(0);
            refresh_ids();
            combine(c);
            if (more) stage_xz(c + 1);
            __syncthreads();
        }
    }
}

// Both moment-gradient scans in one launch: blocks [0, 4BH) build dq^ (chunks
// in order), blocks [4BH, 8BH) build dk^ (chunks in reverse order).
template <bool CAUSAL>
__global__ __launch_bounds__(MG_NTH, 1) void bwd_mg_scans(const _Float16 *__restrict__ qh,
                                                          const _Float16 *__restrict__ kh,
                                                          const bf16_t *__restrict__ v,
                                                          const bf16_t *__restrict__ dout,
                                                          const float *__restrict__ rg,
                                                          const float *__restrict__ cc,
                                                          const float *__restrict__ hmax,
                                                          float *__restrict__ dqh,
                                                          float *__restrict__ dkh, int N, int BH)
{
    extern __shared__ __align__(16) unsigned char smem_raw[];
    GSmem &sm = *reinterpret_cast<GSmem *>(smem_raw);
    const int half = 4 * BH;
    const int b = blockIdx.x;
    if (b < half)
        mg_scan<0, CAUSAL>(sm, b, half, qh, kh, dout, v, rg, cc, hmax, dqh, N, BH);
    else
        mg_scan<1, CAUSAL>(sm, b - half, half, kh, qh, v, dout, rg, cc, hmax, dkh, N, BH);
}

// dv and the in-chunk pairs in one launch: blocks [0, ndv) run the causal scan
// in reverse for dv (fm_causal_scan.h; ndv = 4BH, or 8BH when the scan is
// split into two segments), the rest are the in-chunk blocks (head, chunk).
// The short in-chunk blocks come last and fill the CUs the dv blocks leave
// idle in their last, partly filled round.
__global__ __launch_bounds__(512, 2) void bwd_dv_intra(const _Float16 *__restrict__ qh,
                                                       const _Float16 *__restrict__ kh,
                                                       const bf16_t *__restrict__ v,
                                                       const bf16_t *__restrict__ dout,
                                                       const float *__restrict__ rg,
                                                       const float *__restrict__ cc,
                                                       const float *__restrict__ hmax,
                                                       float *__restrict__ dqh,
                                                       float *__restrict__ dkh,
                                                       bf16_t *__restrict__ dv, int N, int nch,
                                                       int BH, mfma_causal::SegArgs sa)
{
    static_assert(mfma_causal::NTH == 512, "one block size for both");
    extern __shared__ __align__(16) unsigned char smem_raw[];
    const int ndv = 4 * BH * (1 + sa.split);
    const int b = blockIdx.x;
    if (b < ndv) {
        // queries of the dv scan are the keys k^ (and vice versa), values dO / G
        mfma_causal::Smem &sm = *reinterpret_cast<mfma_causal::Smem *>(smem_raw);
        mfma_causal::scan_block<true>(sm, kh, qh, dout, dv, nullptr, rg, N, BH, b, 4 * BH, sa);
    } else {
        ISmem &sm = *reinterpret_cast<ISmem *>(smem_raw);
        intra_block(sm, qh, kh, v, dout, rg, cc, hmax, dqh, dkh, N, nch, b - ndv);
    }
}

// ---------------------------------------------------------------------------
// bwd_finish: dx = (dx^ - mean dx^ - x^ mean(dx^ x^)) / std, an octet per row.

__global__ __launch_bounds__(256) void bwd_finish(const bf16_t *__restrict__ q,
                                                  const bf16_t *__restrict__ k,
                                                  const float *__restrict__ dqh,
                                                  const float *__restrict__ dkh,
                                                  bf16_t *__restrict__ dq, bf16_t *__restrict__ dk,
                                                  size_t rows, float qs)
{
    const size_t r = (size_t)blockIdx.x * 32 + (threadIdx.x >> 3);
    const int cg = threadIdx.x & 7;
    const bool valid = r < rows;
    for (int which = 0; which < 2; ++which) {
        const bf16_t *xs = which ? k : q;
        const float *dh = which ? dkh : dqh;
        bf16_t *dx = which ? dk : dq;
        float xv[8] = {}, d[8] = {};
        if (valid) {
            bf16x8_to_f32(*(const uint4 *)(xs + r * D + 8 * cg), xv);
            const f4 a = *(const f4 *)(dh + r * D + 8 * cg);
            const f4 bq = *(const f4 *)(dh + r * D + 8 * cg + 4);
            // the scans differentiate with respect to the scaled query qs q^
            const float sc = which ? 1.0f : qs;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                d[i] = a[i] * sc;
                d[4 + i] = bq[i] * sc;
            }
        }
        float s = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) s += xv[i];
        const float mu = octet_sum(s) * (1.0f / D);
        float var = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            xv[i] -= mu;
            var = fmaf(xv[i], xv[i], var);
        }
        const float rs = valid ? __builtin_amdgcn_rsqf(octet_sum(var) * (1.0f / D)) : 0.f;
        float m1 = 0.f, m2 = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            xv[i] *= rs;
            m1 += d[i];
            m2 = fmaf(d[i], xv[i], m2);
        }
        m1 = octet_sum(m1) * (1.0f / D);
        m2 = octet_sum(m2) * (1.0f / D);
        if (valid) {
            uint4 o;
            uint32_t *ow = (uint32_t *)&o;
#pragma unroll
            for (int i = 0; i < 4; ++i)
                ow[i] = pack_bf16x2((d[2 * i] - m1 - xv[2 * i] * m2) * rs,
                                    (d[2 * i + 1] - m1 - xv[2 * i + 1] * m2) * rs);
            *(uint4 *)(dx + r * D + 8 * cg) = o;
        }
    }
}

}  // namespace mfma_bwd

namespace mfma_bwd {

size_t base_workspace(int BH, int N)
{
    const size_t rows = (size_t)BH * N;
    auto a256 = [](size_t x) { return (x + 255) & ~(size_t)255; };
    const size_t nch = ((size_t)N + C - 1) / C;
    return a256(rows * 4) * 2 + a256((size_t)BH * nch * 16) + 2 * a256(rows * mx::D * 4) +
           2 * a256(rows * mx::D * 2) + causal_scan_seg_workspace(4 * BH, (int)nch);
}

// Causal: dv by the reverse scan with the in-chunk blocks, then the
// moment-gradient scans over earlier chunks.  Non-causal: dv by the
// non-causal forward kernels (queries and keys exchanged, no divide; their
// workspace after the backward's own), then the moment-gradient scans
// against the totals.
template <bool CAUSAL>
hipError_t run(const void *q, const void *k, const void *v, const void *o, const void *dout,
               const float *g, void *dq, void *dk, void *dv, int BH, int N, float qs, void *ws,
               hipStream_t st)
{
    static_assert(sizeof(ISmem) <= 160 * 1024 && sizeof(GSmem) <= 160 * 1024 &&
                      sizeof(mfma_causal::Smem) <= 160 * 1024,
                  "LDS budget");
    const size_t rows = (size_t)BH * N;
    const int nch = (N + C - 1) / C;
    // the dv scan's split (causal)
    const ScanSplit plan = CAUSAL ? causal_scan_split(4 * BH, nch, false) : ScanSplit{0, 0, 1};
    // prep, dv with the in-chunk blocks, the moment-gradient scans, finish;
    // non-causal: the dv launches
    if (!grid_fits((long long)BH * nch, 256) ||
        (CAUSAL && !grid_fits((long long)BH * (4 * (1 + plan.split) + nch), 512)) ||
        !grid_fits((long long)BH * 8, MG_NTH) || !grid_fits((long long)((rows + 31) / 32), 256) ||
        (!CAUSAL && !mfma_nc_grids_fit(BH, N)))
        return hipErrorInvalidConfiguration;
    auto a256 = [](size_t x) { return (x + 255) & ~(size_t)255; };
    unsigned char *p = (unsigned char *)ws;
    float *rg = (float *)p;
    p += a256(rows * 4);
    float *cc = (float *)p;
    p += a256(rows * 4);
    float *hmax = (float *)p;
    p += a256((size_t)BH * nch * 16);
    float *dqh = (float *)p;
    p += a256(rows * D * 4);
    float *dkh = (float *)p;
    p += a256(rows * D * 4);
    _Float16 *qh = (_Float16 *)p;
    p += a256(rows * D * 2);
    _Float16 *kh = (_Float16 *)p;
    p += a256(rows * D * 2);
    // the dv scan's segment summaries and flags (causal)
    mfma_causal::SegArgs sa{nullptr, nullptr, plan.split, plan.csplit, plan.wait};
    if (plan.split) {
        sa.sum = p;
        sa.flags = (unsigned int *)(p + a256((size_t)4 * BH * mfma_causal::SUM_BYTES));
    }
    p += causal_scan_seg_workspace(4 * BH, nch);

    const bf16_t *Q = (const bf16_t *)q, *K = (const bf16_t *)k, *V = (const bf16_t *)v;
    const bf16_t *O = (const bf16_t *)o, *DO = (const bf16_t *)dout;
    hipLaunchKernelGGL(bwd_prep, dim3(BH * nch), dim3(256), 0, st, Q, K, O, DO, V, g, rg, cc, hmax,
                       qh, kh, N, nch, qs, sa.flags, plan.split ? 4 * BH : 0);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if constexpr (CAUSAL) {
        const size_t smem1 = sizeof(ISmem) > sizeof(mfma_causal::Smem) ? sizeof(ISmem)
                                                                        : sizeof(mfma_causal::Smem);
        e = hipFuncSetAttribute((const void *)bwd_dv_intra,
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem1);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(bwd_dv_intra, dim3(BH * 4 * (1 + plan.split) + BH * nch), dim3(512),
                           smem1, st, qh, kh, V, DO, rg, cc, hmax, dqh, dkh, (bf16_t *)dv, N, nch,
                           BH, sa);
    } else {
        e = mfma_nc_dv(qh, kh, DO, rg, dv, BH, N, p, st);
    }
    e = e == hipSuccess ? hipGetLastError() : e;
    if (e != hipSuccess) return e;
    e = hipFuncSetAttribute((const void *)bwd_mg_scans<CAUSAL>,
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)sizeof(GSmem));
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(bwd_mg_scans<CAUSAL>, dim3(BH * 8), dim3(MG_NTH), sizeof(GSmem), st, qh, kh,
                       V, DO, rg, cc, hmax, dqh, dkh, N, BH);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(bwd_finish, dim3((unsigned)((rows + 31) / 32)), dim3(256), 0, st, Q, K,
                       dqh, dkh, (bf16_t *)dq, (bf16_t *)dk, rows, qs);
    return hipGetLastError();
}

}  // namespace mfma_bwd

size_t mfma_causal_bwd_workspace(int BH, int N) { return mfma_bwd::base_workspace(BH, N); }

hipError_t mfma_causal_bwd(const void *q, const void *k, const void *v, const void *o,
                           const void *dout, const float *g, void *dq, void *dk, void *dv, int BH,
                           int N, float qs, void *ws, hipStream_t st)
{
    return mfma_bwd::run<true>(q, k, v, o, dout, g, dq, dk, dv, BH, N, qs, ws, st);
}

size_t mfma_nc_bwd_workspace(int BH, int N)
{
    return mfma_bwd::base_workspace(BH, N) + mfma_nc_workspace(BH, N);
}

hipError_t mfma_nc_bwd(const void *q, const void *k, const void *v, const void *o,
                       const void *dout, const float *g, void *dq, void *dk, void *dv, int BH,
                       int N, float qs, void *ws, hipStream_t st)
{
    return mfma_bwd::run<false>(q, k, v, o, dout, g, dq, dk, dv, BH, N, qs, ws, st);
}

}  // namespace fm

// Non-causal Fastmax forward on CDNA4 MFMA, head dimension 64, p = 2, bf16 I/O.
//
// The factorised form of Sec. 2.3 (Eqs. "x", "y", "f", "g"): the moments
// S = Phi(K^)^T V (x^1, x^2, x^3), y^2 = sum_n k^_n and Y3 = sum_n k^_n k^_n^T
// (y^3) are built once per head and contracted against Psi(q^_i) for every
// query; y^1 = N.  Three kernels, all on the tile pattern of fm_mfma.h:
//
//  nc_moments (head, 32-column slice, token segment).  Eight waves hold the
//     segment's partial state S[f][j] for 32 value columns as fp32 MFMA
//     accumulators (21 tiles x 2 column tiles per wave); per 32-token K step
//     A = K^T tiles (read once, used for both column tiles) and
//     B = diag(k_m) V generated with packed fp16 multiplies.  v is scaled by
//     a power of two from the segment's max|v| so that the fp16 products
//     stay finite; the partial state is written unscaled in fp32.
//  nc_reduce  sums the segments, applies the 1/2 of the diagonal tiles and a
//     power-of-two scale per 16-column tile (from the bound
//     |S[f][j]| <= 63 sum_n |v_nj|), and writes the fp16 state in the
//     per-lane A-operand order of nc_query; also Y3 (fp16, scaled), y2, x1.
//  nc_query   (head, token block).  All 64 value columns per workgroup: the
//     fp16 state is loaded once into registers (44 A operands per lane), each
//     generated Psi(q) operand feeds four MFMAs (one per 16-column tile).
//     Cross-wave partial F^T are double-buffered in LDS and combined one
//     32-token step behind, with G = N + q.y2 + 1/2 q^T Y3 q (Y3 on MFMA).
#include <hip/hip_runtime.h>

#include <limits.h>

#include "fm_common.h"
#include "fm_internal.h"
#include "fm_mfma.h"

namespace fm {
namespace mfma_nc {

using namespace mx;

constexpr int C = 128;               // tokens per chunk of the moment build
constexpr int NW = 8;                // waves per workgroup
constexpr int NTH = NW * 64;
constexpr int MSW = 32;              // value columns per moment workgroup
constexpr int MCT = MSW / 16;        // column tiles per moment workgroup
constexpr int NMS = D / MSW;         // moment slices per head
constexpr int NCT = D / 16;          // column tiles of a head
constexpr int QS = 32;               // tokens per query step
constexpr int TARGET_BLOCKS = 256;   // workgroups per launch: one per CU of an MI355X
constexpr int HDR = 160;             // floats of the per-head header
// header: [0,64) y2 * 2^(1-gexp); [64,128) x1 * 2^-es(tile); [128,132) 2^es(tile);
// [132] 1/2 * 2^gexp
constexpr int STATE_TILE_F = 256;                      // floats of one 16x16 tile
constexpr int WAVE_STATE_F = NT * STATE_TILE_F;        // one wave, one column tile

struct Plan {
    int nch, nseg, cps, tb, ntb;
    size_t off_part, off_vmx, off_y3p, off_y2p, off_x1p, off_aq, off_y3h, off_hdr, total;
};

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

Plan make_plan(int BH, int N)
{
    Plan P;
    P.nch = (N + C - 1) / C;
    const long long per = (long long)BH * NMS;
    long long want = (TARGET_BLOCKS + per - 1) / per;
    if (want < 1) want = 1;
    if (want > P.nch) want = P.nch;
    P.cps = (int)((P.nch + want - 1) / want);
    P.nseg = (P.nch + P.cps - 1) / P.cps;   // every segment holds at least one chunk
    long long tb = ((long long)N * BH + TARGET_BLOCKS - 1) / TARGET_BLOCKS;
    tb = (tb + QS - 1) / QS * QS;
    const long long nmax = ((long long)N + QS - 1) / QS * QS;
    if (tb > nmax) tb = nmax;
    if (tb < QS) tb = QS;
    P.tb = (int)tb;
    P.ntb = (int)((N + tb - 1) / tb);
    const size_t bh = (size_t)BH, ns = (size_t)P.nseg;
    size_t o = 0;
    P.off_part = o; o = align256(o + bh * NCT * ns * NW * WAVE_STATE_F * sizeof(float));
    P.off_vmx = o;  o = align256(o + bh * NMS * ns * sizeof(float));
    P.off_y3p = o;  o = align256(o + bh * ns * D * D * sizeof(float));
    P.off_y2p = o;  o = align256(o + bh * ns * D * sizeof(float));
    P.off_x1p = o;  o = align256(o + bh * ns * D * sizeof(float));
    P.off_aq = o;   o = align256(o + bh * NW * NKS * NCT * 64 * 16);
    P.off_y3h = o;  o = align256(o + bh * D * D * sizeof(_Float16));
    P.off_hdr = o;  o = align256(o + bh * HDR * sizeof(float));
    P.total = o;
    return P;
}

// ---------------------------------------------------------------------------
// nc_moments

struct MSmem {
    _Float16 kT[2][D * RS128];      // k^ [m][token], double-buffered by chunk parity
    _Float16 vT[2][MSW * RS128];    // scaled v [j][token]
    float red[NW];
};

// KF16: the keys arrive standardised in fp16 (else bf16 rows, standardised
// here).  The backward's dv (Sec. 2.5: dv_n = sum_i f(s_in) u_i, the forward
// with queries and keys exchanged) uses KF16 with the standardised queries
// as keys and the values u_i = dO_i / G_i: each value row v_n is multiplied
// by vrow[n] when vrow is given.
template <bool KF16>
__global__ __launch_bounds__(NTH, 2) void nc_moments(const void *__restrict__ kin,
                                                     const bf16_t *__restrict__ v,
                                                     const float *__restrict__ vrow,
                                                     float *__restrict__ part,
                                                     float *__restrict__ vmx,
                                                     float *__restrict__ y3p,
                                                     float *__restrict__ y2p,
                                                     float *__restrict__ x1p, int N, int BH,
                                                     int nseg, int cps)
{
    __shared__ MSmem sm;

    // Block -> (head, slice, segment).  The slices of one (head, segment) are
    // kept on one XCD (block ids go round-robin over the 8 XCDs) so that its k
    // rows are read from HBM once and shared through that XCD's L2.
    const int nblk = gridDim.x, b = blockIdx.x;
    int sl, rest;
    if ((nblk & 15) == 0) {
        const int xcd = b & 7, idx = b >> 3;
        sl = idx & (NMS - 1);
        rest = (idx / NMS) * 8 + xcd;
    } else {
        sl = b % NMS;
        rest = b / NMS;
    }
    const int head = rest / nseg, seg = rest % nseg;
    if (head >= BH) return;
    const int nch = (N + C - 1) / C;
    const int c0 = seg * cps, c1 = min(nch, c0 + cps);
    const int t0 = c0 * C, t1 = min(N, c1 * C);
    const uint16_t *k = (const uint16_t *)kin + (size_t)head * N * D;
    v += (size_t)head * N * D;
    if (vrow) vrow += (size_t)head * N;

    const int w = threadIdx.x >> 6;
    const bool has_lin = w < 4;
    const bool do_y3 = sl == 0;   // Y3 and y2 are per head: slice 0 builds them

    // max |v| of this slice over the segment -> power-of-two scale with
    // 8 * max|v| * 2^-e <= 2^15 (|k^_m| <= 8)
    int tid = threadIdx.x;
    float vmax = 0.f;
    // eight loads in flight per thread, not one round trip per row quarter
    constexpr int U = 8;
    for (int p0 = 4 * t0 + tid; p0 < 4 * t1; p0 += U * NTH) {
        uint4 raw[U];
        float rr[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int p = p0 + u * NTH, n = p >> 2, qq = p & 3;
            raw[u] = uint4{0u, 0u, 0u, 0u};
            rr[u] = 1.0f;
            if (p < 4 * t1) {
                raw[u] = *(const uint4 *)(v + (size_t)n * D + MSW * sl + 8 * qq);
                // raw: no arithmetic on a loaded value before all U are issued
                if (vrow) rr[u] = vrow[n];
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            float x[8];
            bf16x8_to_f32(raw[u], x);
            const float ar = fabsf(rr[u]);
#pragma unroll
            for (int i = 0; i < 8; ++i) vmax = fmaxf(vmax, fabsf(x[i]) * ar);
        }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) vmax = fmaxf(vmax, __shfl_xor(vmax, o));
    if ((tid & 63) == 0) sm.red[tid >> 6] = vmax;
    __syncthreads();
    vmax = 0.f;
#pragma unroll
    for (int ww = 0; ww < NW; ++ww) vmax = fmaxf(vmax, sm.red[ww]);
    const int vexp = pow2_exponent(8.0f * vmax);
    const float vscale = ldexpf(1.0f, -vexp);

    f4 acc[MCT][NT];
#pragma unroll
    for (int ct = 0; ct < MCT; ++ct)
#pragma unroll
        for (int t = 0; t < NT; ++t) acc[ct][t] = f4{0.f, 0.f, 0.f, 0.f};
    f4 y3acc[2] = {f4{0.f, 0.f, 0.f, 0.f}, f4{0.f, 0.f, 0.f, 0.f}};
    int y3u[2], y3u2[2];
    y3_tile(w, 0, y3u[0], y3u2[0]);
    y3_tile(w, w < 2 ? 1 : 0, y3u[1], y3u2[1]);
    const int ny3 = y3_count(w);
    float ssum = 0.f;   // running sum of k^ (waves 0-3) or of scaled v (waves 4-5)

    int lane = tid & 63, r16 = lane & 15, h = lane >> 4;
    int tg = tid >> 3, cg = tid & 7;       // k loader: tokens 2tg, 2tg+1, channels 8cg..
    int vt = tid >> 2, vq = tid & 3;       // v loader: token vt, columns 8vq..
    auto refresh_ids = [&]() {
        asm volatile("" : "+v"(tid));
        lane = tid & 63;
        r16 = lane & 15;
        h = lane >> 4;
        tg = tid >> 3;
        cg = tid & 7;
        vt = tid >> 2;
        vq = tid & 3;
    };

    uint4 pk[2], pv;
    float pr = 1.0f;
    auto prefetch = [&](int c) {
        const uint4 z = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int n = c * C + 2 * tg + j;
            pk[j] = z;
            if (n < N) pk[j] = *(const uint4 *)(k + (size_t)n * D + 8 * cg);
        }
        const int nv = c * C + vt;
        pv = z;
        if (nv < N) {
            pv = *(const uint4 *)(v + (size_t)nv * D + MSW * sl + 8 * vq);
            if (vrow) pr = vrow[nv];
        }
    };
    // standardise k rows (Sec. 2.2, Eqs. 6-7), store k^ transposed and the
    // scaled v transposed
    auto stage = [&](int c, int buf) {
        h8 hk[2];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            if constexpr (KF16) {
                hk[j] = __builtin_bit_cast(h8, pk[j]);   // rows past N load as zero
            } else {
                float x[8];
                bf16x8_to_f32(pk[j], x);
                hk[j] = standardise8(x, c * C + 2 * tg + j < N);
            }
        }
#pragma unroll
        for (int i = 0; i < 8; ++i)
            *(h2 *)(sm.kT[buf] + sw128(8 * cg + i, 2 * tg)) = h2{hk[0][i], hk[1][i]};
        float xv[8];
        bf16x8_to_f32(pv, xv);
        const float vs = vrow ? vscale * pr : vscale;
#pragma unroll
        for (int i = 0; i < 8; ++i) sm.vT[buf][sw128(8 * vq + i, vt)] = (_Float16)(xv[i] * vs);
    };

    prefetch(c0);
    stage(c0, 0);
    __syncthreads();

    for (int c = c0; c < c1; ++c) {
        const int buf = (c - c0) & 1;
        const bool more = c + 1 < c1;
        __builtin_amdgcn_sched_barrier(0);
        refresh_ids();
        const _Float16 *kTc = sm.kT[buf];
        const _Float16 *vTc = sm.vT[buf];
        // S += Phi(K)^T V for 32 tokens: both column tiles share the K^T tiles
        // and the k_m rows
        auto ustep = [&](int s) {
            h8 Ak[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) Ak[u] = ld8(kTc + sw128(16 * u + r16, 32 * s + 8 * h));
            h8 Vf[MCT];
#pragma unroll
            for (int ct = 0; ct < MCT; ++ct) Vf[ct] = ld8(vTc + sw128(16 * ct + r16, 32 * s + 8 * h));
            if (has_lin) {
                const h8 Al = ld8(kTc + sw128(16 * w + r16, 32 * s + 8 * h));
#pragma unroll
                for (int ct = 0; ct < MCT; ++ct) acc[ct][0] = mfma(Al, Vf[ct], acc[ct][0]);
            }
            static_for<0, 8>([&](auto ii) {
                constexpr int idx = decltype(ii)::value;
                constexpr int u0 = u0_of(idx);
                constexpr int tf = first_tile(idx);
                const h8 km = ld8(kTc + sw128(w + 8 * idx, 32 * s + 8 * h));
#pragma unroll
                for (int ct = 0; ct < MCT; ++ct) {
                    const h8 Wm = km * Vf[ct];
                    static_for<u0, 4>([&](auto ui) {
                        constexpr int u = decltype(ui)::value;
                        acc[ct][tf + (u - u0)] = mfma(Ak[u], Wm, acc[ct][tf + (u - u0)]);
                    });
                }
            });
            if (do_y3) {
#pragma unroll
                for (int kk = 0; kk < 2; ++kk)
                    if (kk < ny3)
                        y3acc[kk] = mfma(ld8(kTc + sw128(16 * y3u[kk] + r16, 32 * s + 8 * h)),
                                         ld8(kTc + sw128(16 * y3u2[kk] + r16, 32 * s + 8 * h)),
                                         y3acc[kk]);
            }
        };
#pragma unroll 1
        for (int s = 0; s < C / 32 - 1; ++s) ustep(s);
        // the next chunk's loads land behind the last K step
        if (more) prefetch(c + 1);
        ustep(C / 32 - 1);
        // per-lane partial sums of k^ (waves 0-3: channel 16w + r16) and of
        // scaled v (waves 4-5: column 16(w-4) + r16), tokens 32h..32h+31
        if (w < 4) {
#pragma unroll
            for (int cc = 0; cc < 4; ++cc) ssum += hsum8(ld8(kTc + sw128(16 * w + r16, 32 * h + 8 * cc)));
        } else if (w < 4 + MCT) {
#pragma unroll
            for (int cc = 0; cc < 4; ++cc)
                ssum += hsum8(ld8(vTc + sw128(16 * (w - 4) + r16, 32 * h + 8 * cc)));
        }
        if (more) stage(c + 1, buf ^ 1);
        __syncthreads();
    }

    // ---- write the segment's partials (unscaled) ------------------------
    refresh_ids();
    const float oscale = ldexpf(1.0f, vexp);
#pragma unroll
    for (int ct = 0; ct < MCT; ++ct) {
        const int gct = MCT * sl + ct;
        float *dst = part + ((((size_t)head * NCT + gct) * nseg + seg) * NW + w) * WAVE_STATE_F +
                     4 * lane;
#pragma unroll
        for (int t = 0; t < NT; ++t) *(f4 *)(dst + t * STATE_TILE_F) = acc[ct][t] * oscale;
    }
    if (tid == 0) vmx[((size_t)head * NMS + sl) * nseg + seg] = vmax;
    ssum += __shfl_xor(ssum, 16);
    ssum += __shfl_xor(ssum, 32);
    const size_t hs = (size_t)head * nseg + seg;
    if (w < 4) {
        if (do_y3 && h == 0) y2p[hs * D + 16 * w + r16] = ssum;
    } else if (w < 4 + MCT) {
        if (h == 0) x1p[hs * D + MSW * sl + 16 * (w - 4) + r16] = ssum * oscale;
    }
    if (do_y3) {
        // lane: column m = 16 u2 + r16, rows l = 16 u + 4h + i of Y3 (symmetric)
        float *y3 = y3p + hs * D * D;
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            if (kk >= ny3) break;
            const int u = y3u[kk], u2 = y3u2[kk];
            const int m = 16 * u2 + r16;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int l = 16 * u + 4 * h + i;
                y3[l * D + m] = y3acc[kk][i];
                if (u != u2) y3[m * D + l] = y3acc[kk][i];
            }
        }
    }
}

// ---------------------------------------------------------------------------
// nc_reduce

constexpr int RED_BLOCKS = NW * NKS * NCT * 64 / 512;   // 44 state blocks per head

__device__ __forceinline__ int seg_tokens(int seg, int N, int cps)
{
    const int t0 = seg * cps * C;
    return max(0, min(N, t0 + cps * C) - t0);
}

__global__ __launch_bounds__(512) void nc_reduce(const float *__restrict__ part,
                                                 const float *__restrict__ vmx,
                                                 const float *__restrict__ y3p,
                                                 const float *__restrict__ y2p,
                                                 const float *__restrict__ x1p,
                                                 h8 *__restrict__ aq, _Float16 *__restrict__ y3h,
                                                 float *__restrict__ hdr, int N, int nseg,
                                                 int cps)
{
    const int head = blockIdx.x / (RED_BLOCKS + 1), blk = blockIdx.x % (RED_BLOCKS + 1);
    const int tid = threadIdx.x;
    // scale exponent per 16-column tile: 63 sum_n |v_nj| bounds every state entry
    auto tile_exp = [&](int ct) {
        const int sl = ct / MCT;
        float bound = 0.f;
        // unrolled: several loads in flight per wait (a loop of dependent
        // waits would cost one memory round trip per segment)
#pragma unroll 8
        for (int s = 0; s < nseg; ++s)
            bound += (float)seg_tokens(s, N, cps) * vmx[((size_t)head * NMS + sl) * nseg + s];
        return pow2_exponent(63.0f * bound);
    };
    if (blk < RED_BLOCKS) {
        const int i = blk * 512 + tid;
        const int lane = i & 63, ct = (i >> 6) & (NCT - 1), rest = i >> 8;
        const int p = rest % NKS, w = rest / NKS;
        const int ta = 2 * p, tb = 2 * p + 1;
        f4 a = {0.f, 0.f, 0.f, 0.f}, bb = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 8
        for (int s = 0; s < nseg; ++s) {
            const float *src = part + ((((size_t)head * NCT + ct) * nseg + s) * NW + w) * WAVE_STATE_F +
                               4 * lane;
            a += *(const f4 *)(src + ta * STATE_TILE_F);
            if (tb < NT) bb += *(const f4 *)(src + tb * STATE_TILE_F);
        }
        const float sc = ldexpf(1.0f, -tile_exp(ct));
        a *= sc * (is_diag(ta) ? 0.5f : 1.0f);
        bb *= sc * (is_diag(tb) ? 0.5f : 1.0f);
        aq[(((size_t)head * NW + w) * NKS + p) * NCT * 64 + ct * 64 + lane] = cat(cvt4(a), cvt4(bb));
    } else {
        const int gexp = max(0, pow2_exponent(64.0f * (float)N));
        const float gs = ldexpf(1.0f, -gexp);
        for (int e = tid; e < D * D; e += 512) {
            float s = 0.f;
#pragma unroll 8
            for (int sg = 0; sg < nseg; ++sg) s += y3p[((size_t)head * nseg + sg) * D * D + e];
            y3h[(size_t)head * D * D + e] = (_Float16)(s * gs);
        }
        float *hd = hdr + (size_t)head * HDR;
        if (tid < D) {
            float s = 0.f;
#pragma unroll 8
            for (int sg = 0; sg < nseg; ++sg) s += y2p[((size_t)head * nseg + sg) * D + tid];
            hd[tid] = s * ldexpf(2.0f, -gexp);
        } else if (tid < 2 * D) {
            const int j = tid - D;
            float s = 0.f;
#pragma unroll 8
            for (int sg = 0; sg < nseg; ++sg) s += x1p[((size_t)head * nseg + sg) * D + j];
            hd[D + j] = s * ldexpf(1.0f, -tile_exp(j / 16));
        } else if (tid < 2 * D + NCT) {
            hd[2 * D + (tid - 2 * D)] = ldexpf(1.0f, tile_exp(tid - 2 * D));
        } else if (tid == 2 * D + NCT) {
            hd[2 * D + NCT] = ldexpf(0.5f, gexp);
        }
    }
}

// ---------------------------------------------------------------------------
// nc_query

struct QSmem {
    float fpart[2][NW * NCT * 4 * QS * 4];   // [buf][wave][tile][row quad][token][4]
    float gpart[2][4 * QS];                  // [buf][channel tile][token]
    _Float16 qrow[2][QS * RS64];             // q^ [token][m], double-buffered by step parity
    _Float16 qperm[2][QS * RS64];            // q^ [token][8 (m % 8) + m / 8]: a wave's channels
                                             // m = w + 8 idx are one 16-byte load
    _Float16 y3h[D * RS64];                  // scaled Y3
    float hdr[HDR];
};

// QF16: the queries arrive standardised in fp16 (else bf16 rows,
// standardised here with the score scale).  DIVIDE = false stores the
// numerator F undivided and no G (the backward's dv).
template <bool QF16, bool DIVIDE>
__global__ __launch_bounds__(NTH, 1) void nc_query(const void *__restrict__ qin,
                                                   const h8 *__restrict__ aq,
                                                   const _Float16 *__restrict__ y3g,
                                                   const float *__restrict__ hdrg,
                                                   bf16_t *__restrict__ out,
                                                   float *__restrict__ g, int N, int BH, int tb,
                                                   int ntb, float qs)
{
    extern __shared__ __align__(16) unsigned char smem_raw[];
    QSmem &sm = *reinterpret_cast<QSmem *>(smem_raw);

    // Block -> (head, token block): consecutive blocks of one head share an
    // XCD (and its L2 copy of the head's state).
    const int nblk = gridDim.x, b = blockIdx.x;
    const int gi = (nblk & 7) == 0 ? (b & 7) * (nblk >> 3) + (b >> 3) : b;
    const int head = gi / ntb, tbi = gi % ntb;
    if (head >= BH) return;
    const int tok0 = tbi * tb, tok1 = min(N, tok0 + tb);
    const int nsteps = (tok1 - tok0 + QS - 1) / QS;
    const uint16_t *q = (const uint16_t *)qin + (size_t)head * N * D;
    out += (size_t)head * N * D;
    if (g) g += (size_t)head * N;

    int tid = threadIdx.x;
    const int w = tid >> 6;
    int lane = tid & 63, r16 = lane & 15, h = lane >> 4;
    auto refresh_ids = [&]() {
        asm volatile("" : "+v"(tid));
        lane = tid & 63;
        r16 = lane & 15;
        h = lane >> 4;
    };

    // the head's fp16 state: A operands of this wave for all K steps and tiles
    h8 Ast[NCT][NKS];
    {
        const h8 *src = aq + ((size_t)head * NW + w) * NKS * NCT * 64 + lane;
#pragma unroll
        for (int p = 0; p < NKS; ++p)
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) Ast[ct][p] = src[(p * NCT + ct) * 64];
    }
    for (int e = tid; e < D * D / 8; e += NTH) {
        const int row = e >> 3, c8 = e & 7;
        *(h8 *)(sm.y3h + sw64(row, 8 * c8)) = *(const h8 *)(y3g + (size_t)head * D * D + row * D + 8 * c8);
    }
    if (tid < HDR) sm.hdr[tid] = hdrg[(size_t)head * HDR + tid];

    // q staging: threads < 256, token tid/8 of the step, channels 8(tid%8)..
    uint4 pq = {0u, 0u, 0u, 0u};
    auto prefetch = [&](int s) {
        const int n = tok0 + s * QS + (tid >> 3);
        pq = uint4{0u, 0u, 0u, 0u};
        if (n < tok1) pq = *(const uint4 *)(q + (size_t)n * D + 8 * (tid & 7));
    };
    auto stage = [&](int s, int buf) {
        const int row = tid >> 3, cg = tid & 7;
        h8 hq;
        if constexpr (QF16) {
            hq = __builtin_bit_cast(h8, pq);   // rows past the block load as zero
        } else {
            float x[8];
            bf16x8_to_f32(pq, x);
            hq = standardise8(x, tok0 + s * QS + row < tok1, qs);
        }
        *(h8 *)(sm.qrow[buf] + sw64(row, 8 * cg)) = hq;
#pragma unroll
        for (int i = 0; i < 8; ++i) sm.qperm[buf][sw64(row, 8 * i + cg)] = hq[i];
    };
    const float Nf = (float)N;
    auto combine = [&](int s) {
        const int buf = s & 1;
        const int tk = tid & (QS - 1), cq = tid >> 5;   // token, column quad 0..15
        const int ct = cq >> 2, hq = cq & 3;
        const int n = tok0 + s * QS + tk;
        f4 F = *(const f4 *)(sm.hdr + D + 4 * cq);
#pragma unroll
        for (int ww = 0; ww < NW; ++ww)
            F += *(const f4 *)(sm.fpart[buf] + (((ww * NCT + ct) * 4 + hq) * QS + tk) * 4);
        float gq = 0.f;
#pragma unroll
        for (int k = 0; k < 4; ++k) gq += sm.gpart[buf][k * QS + tk];
        const float G = fmaf(sm.hdr[2 * D + NCT], gq, Nf);
        if (n < tok1) {
            const float sc = DIVIDE ? sm.hdr[2 * D + ct] * __builtin_amdgcn_rcpf(G) : sm.hdr[2 * D + ct];
            uint2 o;
            o.x = pack_bf16x2(F[0] * sc, F[1] * sc);
            o.y = pack_bf16x2(F[2] * sc, F[3] * sc);
            *(uint2 *)(out + (size_t)n * D + 4 * cq) = o;
            if (DIVIDE && g && cq == 0) g[n] = G;
        }
    };

    if (tid < 256) {
        prefetch(0);
        stage(0, 0);
    }
    __syncthreads();

    for (int s = 0; s < nsteps; ++s) {
        const int buf = s & 1;
        const bool more = s + 1 < nsteps;
        __builtin_amdgcn_sched_barrier(0);
        refresh_ids();
        if (more && tid < 256) prefetch(s + 1);
        const _Float16 *qr = sm.qrow[buf];
#pragma unroll
        for (int rt = 0; rt < QS / 16; ++rt) {
            const int tk = 16 * rt + r16;
            h4 myl[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) myl[u] = ld4(qr + sw64(tk, 16 * u + 4 * h));
            const h4 mylin = ld4(qr + sw64(tk, 16 * (w & 3) + 4 * h));
            const h8 qm = ld8(sm.qperm[buf] + sw64(tk, 8 * w));
            f4 F[NCT];
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) F[ct] = f4{0.f, 0.f, 0.f, 0.f};
            auto gen = [&](auto ti) -> h4 {
                constexpr int t = decltype(ti)::value;
                constexpr Tile T = tile_of(t < NT ? t : 0);
                if constexpr (t >= NT) {
                    return h4{0, 0, 0, 0};
                } else if constexpr (T.kind == 0) {
                    return mylin;
                } else {
                    return scale4(myl[T.u], qm[T.idx]);
                }
            };
            static_for<0, NKS>([&](auto pi) {
                constexpr int p = decltype(pi)::value;
                const h8 B = cat(gen(std::integral_constant<int, 2 * p>{}),
                                 gen(std::integral_constant<int, 2 * p + 1>{}));
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) F[ct] = mfma(Ast[ct][p], B, F[ct]);
            });
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct)
                *(f4 *)(sm.fpart[buf] + (((w * NCT + ct) * 4 + h) * QS + tk) * 4) = F[ct];
            if (rt == (w >> 2)) {
                // denominator part of channel tile cc: q_l (y2_l + (Y3 q)_l), l in tile cc
                const int cc = w & 3;
                f4 T;
#pragma unroll
                for (int i = 0; i < 4; ++i) T[i] = sm.hdr[16 * cc + 4 * h + i];
                T = mfma(ld8(sm.y3h + sw64(16 * cc + r16, 8 * h)), ld8(qr + sw64(tk, 8 * h)), T);
                T = mfma(ld8(sm.y3h + sw64(16 * cc + r16, 32 + 8 * h)), ld8(qr + sw64(tk, 32 + 8 * h)), T);
                const h4 ql = ld4(qr + sw64(tk, 16 * cc + 4 * h));
                float gq = 0.f;
#pragma unroll
                for (int i = 0; i < 4; ++i) gq = fmaf((float)ql[i], T[i], gq);
                // summed over the four lane groups here, so the combine reads
                // one value per channel tile instead of four
                gq = rows4_sum(gq);
                if (h == 0) sm.gpart[buf][cc * QS + tk] = gq;
            }
        }
        if (s > 0) combine(s - 1);
        if (more && tid < 256) stage(s + 1, buf ^ 1);
        __syncthreads();
    }
    combine(nsteps - 1);
}

}  // namespace mfma_nc

size_t mfma_nc_workspace(int BH, int N) { return mfma_nc::make_plan(BH, N).total; }

bool mfma_nc_grids_fit(int BH, int N)
{
    using namespace mfma_nc;
    const Plan P = make_plan(BH, N);
    return grid_fits((long long)BH * NMS * P.nseg, NTH) &&
           grid_fits((long long)BH * (RED_BLOCKS + 1), 512) && grid_fits((long long)BH * P.ntb, NTH);
}

namespace mfma_nc {

// The three launches on a workspace laid out by make_plan.  KQF16: keys and
// queries arrive standardised in fp16; vrow: per-row value scale (nullptr:
// none); DIVIDE: O = F / G (else F).
template <bool KQF16, bool DIVIDE>
hipError_t launch(const void *q, const void *k, const void *v, const float *vrow, void *out,
                  float *g, int BH, int N, float qs, void *ws, hipStream_t st)
{
    static_assert(sizeof(QSmem) <= 160 * 1024, "LDS budget");
    const Plan P = make_plan(BH, N);
    const long long gm = (long long)BH * NMS * P.nseg;
    const long long gr = (long long)BH * (RED_BLOCKS + 1);
    const long long gq = (long long)BH * P.ntb;
    if (!mfma_nc_grids_fit(BH, N)) return hipErrorInvalidConfiguration;
    unsigned char *w = (unsigned char *)ws;
    float *part = (float *)(w + P.off_part);
    float *vmx = (float *)(w + P.off_vmx);
    float *y3p = (float *)(w + P.off_y3p);
    float *y2p = (float *)(w + P.off_y2p);
    float *x1p = (float *)(w + P.off_x1p);
    h8 *aq = (h8 *)(w + P.off_aq);
    _Float16 *y3h = (_Float16 *)(w + P.off_y3h);
    float *hdr = (float *)(w + P.off_hdr);

    hipLaunchKernelGGL(nc_moments<KQF16>, dim3((unsigned)gm), dim3(NTH), 0, st, k,
                       (const bf16_t *)v, vrow, part, vmx, y3p, y2p, x1p, N, BH, P.nseg, P.cps);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(nc_reduce, dim3((unsigned)gr), dim3(512), 0, st, part, vmx, y3p, y2p, x1p,
                       aq, y3h, hdr, N, P.nseg, P.cps);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const size_t smem = sizeof(QSmem);
    e = hipFuncSetAttribute((const void *)nc_query<KQF16, DIVIDE>,
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((nc_query<KQF16, DIVIDE>), dim3((unsigned)gq), dim3(NTH), smem, st, q, aq,
                       y3h, hdr, (bf16_t *)out, g, N, BH, P.tb, P.ntb, qs);
    return hipGetLastError();
}

}  // namespace mfma_nc

hipError_t mfma_nc_fwd(const void *q, const void *k, const void *v, void *out, float *g, int BH,
                       int N, float qs, void *ws, hipStream_t st)
{
    return mfma_nc::launch<false, true>(q, k, v, nullptr, out, g, BH, N, qs, ws, st);
}

// dv_n = sum_i f(qs q^_i . k^_n) u_i, u_i = dO_i / G_i (Sec. 2.5), over all
// i: the non-causal forward with queries and keys exchanged (keys qs q^,
// queries k^, both standardised in fp16), values dO scaled per row by 1/G,
// and no divide.
hipError_t mfma_nc_dv(const void *qh, const void *kh, const void *dout, const float *rg, void *dv,
                      int BH, int N, void *ws, hipStream_t st)
{
    return mfma_nc::launch<true, false>(kh, qh, dout, rg, dv, nullptr, BH, N, 1.0f, ws, st);
}

}  // namespace fm

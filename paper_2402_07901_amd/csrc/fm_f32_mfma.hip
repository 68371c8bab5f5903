// Fastmax forward on float32 MFMA (v_mfma_f32_16x16x4_f32), p = 2,
// D in {16, 32, 64}, causal and non-causal, float32 or bf16 I/O (the bf16,
// D = 64 cases have their own fp16 kernels).  Every product and sum is fp32,
// so the results meet the float32 bar.
//
// The factorisation of Sec. 2.4: per (head, 16-column slice of V) the moment
// state S[f][j] = sum_n phi_f(k^_n) v_nj over the features
// phi = [k_l, (k_m k_l)] (the constant feature is x1 = sum_n v_n) is held in
// MFMA accumulators (fp32) and contracted against psi(q^) (Eqs. "f", "g");
// the denominator G_i = n + q^.y2 + 1/2 q^T Y3 q^ (y2 = sum k^, Y3 = sum k^k^T)
// is a second, small contraction.  Causal rows add the in-chunk block
// tril(f(Q^K^T))V of their 32-token chunk (Eqs. "xcausal", "ycausal" carried
// across chunks).
//
// Feature tiles (16 features x 16 value columns, one fp32 accumulator per
// lane and row quad): the linear tiles u (features k_l, l = 16u..16u+15) and
// the quadratic tiles (m, u) for u >= m/16 (features k_m k_l): the diagonal
// tiles u = m/16 hold both (m, l) and (l, m) and enter the query contraction
// with weight 1/2, so psi(q).phi(k) = s + s^2/2.  Wave w owns the linear
// tile u = w (w < D/16) and every quadratic tile of the channels
// m = w + 4c: D/4 channels, 4 (D/16)(D/16 + 1)/2 tiles.
//
// MFMA lane layout (16x16x4 f32, lane = 16h + r16): A holds row r16, K index
// h; B holds column r16, K index h; the accumulator holds column r16, rows
// 4h..4h+3.  Contractions over 16 features run as four K steps i = 0..3 with
// K index h <-> feature 4h + i, so element i of a state accumulator is
// directly the A operand of step i (no data movement).
//
// Segments (few heads): a sequence is cut into segments of whole chunks.
// seg kernel (DELTA): each segment's moment sums, all in parallel; prefix
// kernel: their exclusive prefix in place (causal) or the total (non-causal);
// scan kernel: each segment's chunks from that state (causal: queries,
// in-chunk block and state update; non-causal: queries against the total).
// With one segment per (head, slice) a single launch does it all (non-causal:
// the totals over every chunk, then every query; mode BOTH) and no workspace
// is needed.
#include <hip/hip_runtime.h>

#include <limits.h>

#include "fm_common.h"
#include "fm_internal.h"
#include "fm_mfma.h"

namespace fm {
namespace m32 {

using mx::static_for;
typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int C = 32;      // tokens per chunk
constexpr int NW = 4;      // waves
constexpr int NTH = NW * 64;
constexpr int SL = 16;     // value columns per workgroup
constexpr int TARGET_BLOCKS = 256;

__device__ __forceinline__ f4 mma(float a, float b, f4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

template <int D>
struct Pat {
    static constexpr int NU = D / 16;                  // 16-channel blocks
    static constexpr int NCH = D / 4;                  // channels per wave
    static constexpr int NQ = 4 * NU * (NU + 1) / 2;   // quadratic tiles per wave
    static constexpr int NT = 1 + NQ;                  // + the linear slot
    static constexpr int NY3 = NU * (NU + 1) / 2;      // Y3 tiles (u <= u2)
    // first tile of channel c (its diagonal tile; u runs from c/4 to NU-1)
    static constexpr int first(int c)
    {
        int t = 1;
        for (int cc = 0; cc < c; ++cc) t += NU - cc / 4;
        return t;
    }
    static constexpr int RS = D + 2;   // row stride of row-major tiles (floats)
    static constexpr int TS = C + 2;   // row stride of transposed tiles
};

template <int D>
struct Smem {
    float qrow[C * Pat<D>::RS];     // q^ (times the score scale) [token][channel]
    float krow[C * Pat<D>::RS];     // k^ [token][channel]
    float kT[D * Pat<D>::TS];       // k^ [channel][token]
    float vrow[C * SL];             // v slice [token][column]
    float y3[D * Pat<D>::RS];       // Y3 prefix (before the chunk)
    float y2s[D];                   // 2 y2 prefix
    float x1[SL];                   // x1 prefix
    f4 fpart[NW][C / 16][64];       // partial F^T of the waves
    float gin[C];                   // in-chunk row sums
    float gint[NW][C];              // partial q^T(Y3 q^ + 2 y2) per l block
};

// summary of a segment: [wave][tile][lane] f4 state, Y3 [D][D], y2 [D], x1 [SL]
template <int D>
struct Sum {
    static constexpr size_t STATE = (size_t)NW * Pat<D>::NT * 64 * 4;
    static constexpr size_t FLOATS = STATE + (size_t)D * D + D + SL;
    static constexpr size_t BYTES = (FLOATS * 4 + 255) & ~(size_t)255;
};

enum Mode { DELTA = 0, SCAN = 1, QUERY = 2, BOTH = 3 };

// Standardises the D/8 channels [8 lanes per token] this thread holds
// (Sec. 2.2, Eqs. 6-7: population std, no epsilon) and scales them.
template <int D>
__device__ __forceinline__ void standardise_part(float (&x)[D / 8], bool valid, float scale)
{
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < D / 8; ++i) s += x[i];
    s += __shfl_xor(s, 1);
    s += __shfl_xor(s, 2);
    s += __shfl_xor(s, 4);
    const float mu = s * (1.0f / D);
    float v = 0.f;
#pragma unroll
    for (int i = 0; i < D / 8; ++i) {
        x[i] -= mu;
        v = fmaf(x[i], x[i], v);
    }
    v += __shfl_xor(v, 1);
    v += __shfl_xor(v, 2);
    v += __shfl_xor(v, 4);
    const float r = valid ? __builtin_amdgcn_rsqf(v * (1.0f / D)) * scale : 0.0f;
#pragma unroll
    for (int i = 0; i < D / 8; ++i) x[i] *= r;
}

// One workgroup: (item = head * NSL + slice, segment).
template <int D, typename T, bool CAUSAL, int MODE>
__global__ __launch_bounds__(NTH) void scan_kernel(const T *__restrict__ q, const T *__restrict__ k,
                                                   const T *__restrict__ v, T *__restrict__ out,
                                                   float *__restrict__ g, float *__restrict__ sums,
                                                   int N, int nseg, float qs)
{
    using PT = Pat<D>;
    constexpr int NU = PT::NU, NCH = PT::NCH, NT = PT::NT, RS = PT::RS, TS = PT::TS;
    constexpr int NSL = D / SL;
    __shared__ Smem<D> sm;

    const int item = blockIdx.x / nseg, seg = blockIdx.x % nseg;
    const int head = item / NSL, sl = item % NSL;
    const int nch = (N + C - 1) / C;
    const int cbeg = (int)((long long)seg * nch / nseg), cend = (int)((long long)(seg + 1) * nch / nseg);
    const size_t hb = (size_t)head * N * D;
    q += hb;
    k += hb;
    v += hb;
    out += hb;
    if (g) g += (size_t)head * N;
    float *sum = sums ? sums + (size_t)(item * nseg + seg) * (Sum<D>::BYTES / 4) : nullptr;

    const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, r16 = lane & 15, h = lane >> 4;

    // ---- state, prefix sums and Y3 -------------------------------------
    f4 S[NT];
    const bool loaded = MODE == QUERY || (MODE == SCAN && seg > 0);
#pragma unroll
    for (int t = 0; t < NT; ++t)
        S[t] = loaded ? *(const f4 *)(sum + ((size_t)(w * NT + t) * 64 + lane) * 4) : f4{0.f, 0.f, 0.f, 0.f};
    float y2reg = 0.f, x1reg = 0.f;   // thread d < D: y2[d]; D <= tid < D + SL: x1[tid - D]
    {
        const float *sy3 = loaded ? sum + Sum<D>::STATE : nullptr;
        for (int e = tid; e < D * D; e += NTH) sm.y3[(e / D) * RS + e % D] = loaded ? sy3[e] : 0.f;
        if (tid < D) {
            y2reg = loaded ? sy3[D * D + tid] : 0.f;
            sm.y2s[tid] = 2.0f * y2reg;
        } else if (tid < D + SL) {
            x1reg = loaded ? sy3[D * D + D + (tid - D)] : 0.f;
            sm.x1[tid - D] = x1reg;
        }
    }
    // Y3 accumulator tiles of this wave: tile index yi = w + 4 kk over the
    // pairs (u, u2), u <= u2, in row order
    constexpr int NYW = (PT::NY3 + NW - 1) / NW;
    f4 Y[NYW];
    int yu[NYW], yu2[NYW];
#pragma unroll
    for (int kk = 0; kk < NYW; ++kk) {
        const int yi = w + NW * kk;
        int u = 0, rem = yi;
        while (u < NU && rem >= NU - u) {
            rem -= NU - u;
            ++u;
        }
        yu[kk] = u;
        yu2[kk] = u + rem;
        Y[kk] = f4{0.f, 0.f, 0.f, 0.f};
    }
    __syncthreads();
    if (loaded) {
#pragma unroll
        for (int kk = 0; kk < NYW; ++kk) {
            if (w + NW * kk >= PT::NY3) break;
#pragma unroll
            for (int i = 0; i < 4; ++i) Y[kk][i] = sm.y3[(16 * yu[kk] + 4 * h + i) * RS + 16 * yu2[kk] + r16];
        }
    }

    // ---- staging: token tg = tid / 8, channels 8-way split, 2 v columns -
    const int tg = tid >> 3, part = tid & 7;
    constexpr int DP = D / 8;
    // the next chunk's rows are loaded into registers while the current one
    // is processed
    float pq[DP], pk[DP], pv[2];
    bool pvalid = false;
    auto prefetch = [&](int c) {
        const int n = c * C + tg;
        pvalid = n < N;
#pragma unroll
        for (int i = 0; i < DP; ++i) {
            pq[i] = pvalid ? io<T>::ld(q, (size_t)n * D + part * DP + i) : 0.f;
            pk[i] = pvalid ? io<T>::ld(k, (size_t)n * D + part * DP + i) : 0.f;
        }
#pragma unroll
        for (int i = 0; i < 2; ++i) pv[i] = pvalid ? io<T>::ld(v, (size_t)n * D + SL * sl + 2 * part + i) : 0.f;
    };
    auto stage = [&]() {
        standardise_part<D>(pq, pvalid, qs);
        standardise_part<D>(pk, pvalid, 1.0f);
#pragma unroll
        for (int i = 0; i < DP; ++i) {
            const int ch = part * DP + i;
            sm.qrow[tg * RS + ch] = pq[i];
            sm.krow[tg * RS + ch] = pk[i];
            sm.kT[ch * TS + tg] = pk[i];
        }
#pragma unroll
        for (int i = 0; i < 2; ++i) sm.vrow[tg * SL + 2 * part + i] = pv[i];
    };

    // one chunk in mode M (DELTA: state update only; QUERY: outputs only;
    // SCAN: outputs, then the update unless the segment ends here)
    auto chunk = [&](auto mc, int c) {
        constexpr int M = decltype(mc)::value;
            const int n0 = c * C;
            stage();
            if (c + 1 < cend) prefetch(c + 1);
            __syncthreads();

            if constexpr (M != DELTA) {
                // ---- queries: F^T partials over the wave's tiles -----------
    #pragma unroll
                for (int rt = 0; rt < C / 16; ++rt) {
                    const int tok = 16 * rt + r16;
                    const float *qr = sm.qrow + tok * RS;
                    float ql[NU][4];
    #pragma unroll
                    for (int u = 0; u < NU; ++u)
    #pragma unroll
                        for (int i = 0; i < 4; ++i) ql[u][i] = qr[16 * u + 4 * h + i];
                    f4 F = {0.f, 0.f, 0.f, 0.f};
                    if (w < NU) {
                        const float *qw = qr + 16 * w + 4 * h;
    #pragma unroll
                        for (int i = 0; i < 4; ++i) F = mma(S[0][i], qw[i], F);
                    }
                    static_for<0, NCH>([&](auto ci) {
                        constexpr int cc = decltype(ci)::value;
                        constexpr int u0 = cc / 4;
                        const float qm = qr[w + 4 * cc];
                        static_for<u0, NU>([&](auto ui) {
                            constexpr int u = decltype(ui)::value;
                            constexpr int t = PT::first(cc) + u - u0;
                            const float qmw = (u == u0) ? 0.5f * qm : qm;
    #pragma unroll
                            for (int i = 0; i < 4; ++i) F = mma(S[t][i], qmw * ql[u][i], F);
                        });
                    });
                    if constexpr (M == SCAN && CAUSAL) {
                        // in-chunk block of row tile rt (wave rt): key tiles st <= rt
                        if (w == rt) {
                            float gsum = 0.f;
    #pragma unroll
                            for (int st = 0; st <= rt; ++st) {
                                f4 Sc = {0.f, 0.f, 0.f, 0.f};
                                const float *kr = sm.krow + (16 * st + r16) * RS;
    #pragma unroll
                                for (int kk = 0; kk < D / 4; ++kk) Sc = mma(kr[4 * kk + h], qr[4 * kk + h], Sc);
                                // lane: query tok, keys 16 st + 4h + i
    #pragma unroll
                                for (int i = 0; i < 4; ++i) {
                                    float wv = fmaf(0.5f * Sc[i], Sc[i], 1.0f + Sc[i]);
                                    if (st == rt && 4 * h + i > r16) wv = 0.0f;
                                    Sc[i] = wv;
                                    gsum += wv;
                                }
    #pragma unroll
                                for (int i = 0; i < 4; ++i)
                                    F = mma(sm.vrow[(16 * st + 4 * h + i) * SL + r16], Sc[i], F);
                            }
                            gsum += __shfl_xor(gsum, 16);
                            gsum += __shfl_xor(gsum, 32);
                            if (h == 0) sm.gin[tok] = gsum;
                        }
                    }
                    sm.fpart[w][rt][lane] = F;
                    // denominator: q^T (Y3 q + 2 y2) over l block w
                    if (w < NU) {
                        f4 Tq;
    #pragma unroll
                        for (int i = 0; i < 4; ++i) Tq[i] = sm.y2s[16 * w + 4 * h + i];
                        const float *yr = sm.y3 + (16 * w + r16) * RS;
    #pragma unroll
                        for (int kk = 0; kk < D / 4; ++kk) Tq = mma(yr[4 * kk + h], qr[4 * kk + h], Tq);
                        float gq = 0.f;
    #pragma unroll
                        for (int i = 0; i < 4; ++i) gq = fmaf(qr[16 * w + 4 * h + i], Tq[i], gq);
                        gq += __shfl_xor(gq, 16);
                        gq += __shfl_xor(gq, 32);
                        if (h == 0) sm.gint[w][tok] = gq;
                    }
                }
                __syncthreads();
                // ---- outputs O = F / G: token tg, columns 2 part, 2 part + 1 --
                {
                    const int n = n0 + tg;
                    if (n < N) {
                        const int rt = tg >> 4, t16 = tg & 15;
                        float gsum = 0.f;
    #pragma unroll
                        for (int ww = 0; ww < NU; ++ww) gsum += sm.gint[ww][tg];
                        float G = (M == QUERY ? (float)N : (float)n0) + 0.5f * gsum;
                        if (M == SCAN && CAUSAL) G += sm.gin[tg];
                        const float rG = 1.0f / G;
    #pragma unroll
                        for (int i = 0; i < 2; ++i) {
                            const int j = 2 * part + i;
                            float F = sm.x1[j];
    #pragma unroll
                            for (int ww = 0; ww < NW; ++ww) F += sm.fpart[ww][rt][16 * (j >> 2) + t16][j & 3];
                            io<T>::st(out, (size_t)n * D + SL * sl + j, F * rG);
                        }
                        if (g && sl == 0 && part == 0) g[n] = G;
                    }
                }
            }
            if constexpr (M != QUERY) {
                if (M == SCAN && c + 1 == cend) return;   // the next segment starts from its prefix
                // ---- state update S += Phi(K^)^T V, Y3 += K^T K, y2, x1 --------
                float Ak[NU][C / 4], Vb[C / 4];
    #pragma unroll
                for (int u = 0; u < NU; ++u)
    #pragma unroll
                    for (int ks = 0; ks < C / 4; ++ks) Ak[u][ks] = sm.kT[(16 * u + r16) * TS + 4 * ks + h];
    #pragma unroll
                for (int ks = 0; ks < C / 4; ++ks) Vb[ks] = sm.vrow[(4 * ks + h) * SL + r16];
                if (w < NU) {
                    const float *kl = sm.kT + (16 * w + r16) * TS + h;
    #pragma unroll
                    for (int ks = 0; ks < C / 4; ++ks) S[0] = mma(kl[4 * ks], Vb[ks], S[0]);
                }
                static_for<0, NCH>([&](auto ci) {
                    constexpr int cc = decltype(ci)::value;
                    constexpr int u0 = cc / 4;
                    const float *km = sm.kT + (w + 4 * cc) * TS + h;
                    float Bm[C / 4];
    #pragma unroll
                    for (int ks = 0; ks < C / 4; ++ks) Bm[ks] = km[4 * ks] * Vb[ks];
                    static_for<u0, NU>([&](auto ui) {
                        constexpr int u = decltype(ui)::value;
                        constexpr int t = PT::first(cc) + u - u0;
    #pragma unroll
                        for (int ks = 0; ks < C / 4; ++ks) S[t] = mma(Ak[u][ks], Bm[ks], S[t]);
                    });
                });
    #pragma unroll
                for (int kk = 0; kk < NYW; ++kk) {
                    if (w + NW * kk >= PT::NY3) break;
                    const float *a = sm.kT + (16 * yu[kk] + r16) * TS + h;
                    const float *b = sm.kT + (16 * yu2[kk] + r16) * TS + h;
    #pragma unroll
                    for (int ks = 0; ks < C / 4; ++ks) Y[kk] = mma(a[4 * ks], b[4 * ks], Y[kk]);
                }
                if (tid < D) {
                    float s = 0.f;
    #pragma unroll 8
                    for (int t = 0; t < C; ++t) s += sm.krow[t * RS + tid];
                    y2reg += s;
                } else if (tid < D + SL) {
                    float s = 0.f;
    #pragma unroll 8
                    for (int t = 0; t < C; ++t) s += sm.vrow[t * SL + tid - D];
                    x1reg += s;
                }
                __syncthreads();
                // the prefix after this chunk, for the next chunk's outputs
    #pragma unroll
                for (int kk = 0; kk < NYW; ++kk) {
                    if (w + NW * kk >= PT::NY3) break;
    #pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int l = 16 * yu[kk] + 4 * h + i, m = 16 * yu2[kk] + r16;
                        sm.y3[l * RS + m] = Y[kk][i];
                        sm.y3[m * RS + l] = Y[kk][i];
                    }
                }
                if (tid < D) sm.y2s[tid] = 2.0f * y2reg;
                else if (tid < D + SL) sm.x1[tid - D] = x1reg;
            }
            __syncthreads();
    };
    if constexpr (MODE == BOTH) {
        // non-causal, one segment: the totals first, then every query
        prefetch(cbeg);
        for (int c = cbeg; c < cend; ++c) chunk(std::integral_constant<int, DELTA>{}, c);
        prefetch(cbeg);
        for (int c = cbeg; c < cend; ++c) chunk(std::integral_constant<int, QUERY>{}, c);
    } else {
        prefetch(cbeg);
        for (int c = cbeg; c < cend; ++c) chunk(std::integral_constant<int, MODE>{}, c);
    }

    if constexpr (MODE == DELTA) {
        // this segment's sums: state, Y3 (from LDS, written by the last
        // update), y2, x1
#pragma unroll
        for (int t = 0; t < NT; ++t) *(f4 *)(sum + ((size_t)(w * NT + t) * 64 + lane) * 4) = S[t];
        float *sy3 = sum + Sum<D>::STATE;
        for (int e = tid; e < D * D; e += NTH) sy3[e] = sm.y3[(e / D) * RS + e % D];
        if (tid < D) sy3[D * D + tid] = y2reg;
        else if (tid < D + SL) sy3[D * D + D + (tid - D)] = x1reg;
    }
}

// Segment sums -> exclusive prefix over segments (causal) or the total in
// every segment (non-causal), in place; one thread per float of one item.
__global__ __launch_bounds__(256) void prefix_kernel(float *__restrict__ sums, int nseg,
                                                     size_t floats, size_t stride, int causal)
{
    const size_t f = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (f >= floats) return;
    float *p = sums + (size_t)blockIdx.y * nseg * stride + f;
    // 16 segments' values loaded at a time (one memory latency per batch)
    constexpr int BT = 16;
    float run = 0.f;
    if (!causal) {
        for (int s0 = 0; s0 < nseg; s0 += BT) {
            float d[BT];
#pragma unroll
            for (int b = 0; b < BT; ++b) d[b] = s0 + b < nseg ? p[(size_t)(s0 + b) * stride] : 0.f;
#pragma unroll
            for (int b = 0; b < BT; ++b) run += d[b];
        }
    }
    for (int s0 = 0; s0 < nseg; s0 += BT) {
        float d[BT];
#pragma unroll
        for (int b = 0; b < BT; ++b) d[b] = causal && s0 + b < nseg ? p[(size_t)(s0 + b) * stride] : 0.f;
#pragma unroll
        for (int b = 0; b < BT; ++b) {
            if (s0 + b < nseg) p[(size_t)(s0 + b) * stride] = run;
            if (causal) run += d[b];
        }
    }
}

int nseg_of(int items, int nch)
{
    int s = TARGET_BLOCKS / (items > 0 ? items : 1);
    if (s < 1) s = 1;
    if (s > nch) s = nch;
    return s;
}

template <int D, typename T>
hipError_t run(const void *q, const void *k, const void *v, void *out, float *g, int BH, int N,
               int causal, float qs, void *ws, hipStream_t st)
{
    constexpr int NSL = D / SL;
    const int items = BH * NSL;
    const int nch = (N + C - 1) / C;
    const int nseg = nseg_of(items, nch);
    if ((long long)items * nseg > INT_MAX) return hipErrorInvalidConfiguration;
    const dim3 grid((unsigned)(items * nseg));
    const T *Q = (const T *)q, *K = (const T *)k, *V = (const T *)v;
    float *sums = nseg > 1 ? (float *)ws : nullptr;
    const size_t stride = Sum<D>::BYTES / 4;
    if (causal) {
        if (nseg > 1) {
            hipLaunchKernelGGL((scan_kernel<D, T, true, DELTA>), grid, dim3(NTH), 0, st, Q, K, V,
                               (T *)out, g, sums, N, nseg, qs);
            hipLaunchKernelGGL(prefix_kernel, dim3((unsigned)((Sum<D>::FLOATS + 255) / 256), items),
                               dim3(256), 0, st, sums, nseg, Sum<D>::FLOATS, stride, 1);
        }
        hipLaunchKernelGGL((scan_kernel<D, T, true, SCAN>), grid, dim3(NTH), 0, st, Q, K, V,
                           (T *)out, g, sums, N, nseg, qs);
    } else if (nseg == 1) {
        hipLaunchKernelGGL((scan_kernel<D, T, false, BOTH>), grid, dim3(NTH), 0, st, Q, K, V,
                           (T *)out, g, nullptr, N, nseg, qs);
    } else {
        hipLaunchKernelGGL((scan_kernel<D, T, false, DELTA>), grid, dim3(NTH), 0, st, Q, K, V,
                           (T *)out, g, sums, N, nseg, qs);
        hipLaunchKernelGGL(prefix_kernel, dim3((unsigned)((Sum<D>::FLOATS + 255) / 256), items),
                           dim3(256), 0, st, sums, nseg, Sum<D>::FLOATS, stride, 0);
        hipLaunchKernelGGL((scan_kernel<D, T, false, QUERY>), grid, dim3(NTH), 0, st, Q, K, V,
                           (T *)out, g, sums, N, nseg, qs);
    }
    return hipGetLastError();
}

}  // namespace m32

bool f32mfma_applies(int D, int p, int is_bf16)
{
    return p == 2 && (D == 16 || D == 32 || (D == 64 && !is_bf16));
}

size_t f32mfma_fwd_workspace(int BH, int N, int D)
{
    using namespace m32;
    const int nch = (N + C - 1) / C;
    const int items = BH * (D / SL);
    const int nseg = nseg_of(items, nch);
    if (nseg == 1) return 0;   // one workgroup per (head, slice): no segment sums
    const size_t per = D == 16 ? Sum<16>::BYTES : D == 32 ? Sum<32>::BYTES : Sum<64>::BYTES;
    return (size_t)items * nseg * per;
}

hipError_t f32mfma_fwd(const void *q, const void *k, const void *v, void *out, float *g, int BH,
                       int N, int D, int causal, int is_bf16, float qs, void *ws, hipStream_t st)
{
    using namespace m32;
    if (is_bf16) {
        if (D == 16) return run<16, bf16_t>(q, k, v, out, g, BH, N, causal, qs, ws, st);
        if (D == 32) return run<32, bf16_t>(q, k, v, out, g, BH, N, causal, qs, ws, st);
        return hipErrorInvalidValue;
    }
    if (D == 16) return run<16, float>(q, k, v, out, g, BH, N, causal, qs, ws, st);
    if (D == 32) return run<32, float>(q, k, v, out, g, BH, N, causal, qs, ws, st);
    if (D == 64) return run<64, float>(q, k, v, out, g, BH, N, causal, qs, ws, st);
    return hipErrorInvalidValue;
}

}  // namespace fm

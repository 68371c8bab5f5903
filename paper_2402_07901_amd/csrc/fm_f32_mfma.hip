// Fastmax forward on float32 MFMA (v_mfma_f32_16x16x4_f32): p = 1 and 2,
// D in {16, 32, 64, 128}, causal and non-causal, float32 or bf16 I/O (bf16,
// D = 64, p = 2 has its own fp16 kernels).  Every product and sum is fp32, so
// the results meet the float32 bar.  p = 1 keeps only the linear tiles and
// the denominator n + q^.y2.
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
// with weight 1/2, so psi(q).phi(k) = s + s^2/2.  Eight waves (two per
// SIMD): wave w owns the linear tile u = w (w < D/16) and every quadratic
// tile of the channels m = w + 8c (at D = 128, p = 2 the four workgroups of
// a slice share the channels over their 32 waves gw, four channels each,
// from blocks chosen so that every wave holds 18 quadratic tiles); at most
// 21 tiles per wave.  The query contraction sums S[(m, l)] q^_l over the
// tiles of channel m before it multiplies by q^_m.
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
//
// DV mode: the backward's dv (the same scan over the reversed sequence with
// queries and keys exchanged, values dO/G, no denominator).
#include <hip/hip_runtime.h>

#include <limits.h>

#include "fm_common.h"
#include "fm_internal.h"
#include "fm_f32_mfma.h"

namespace fm {
namespace m32 {

template <int D, int P>
struct Smem {
    float qrow[C * Pat<D, P>::RS];  // q^ (times the score scale) [token][channel]
    float krow[C * Pat<D, P>::RS];  // k^ [token][channel]
    float kT[D * Pat<D, P>::TS];    // k^ [channel][token]
    float vrow[C * SL];             // v slice [token][column]
    float y3[(Pat<D, P>::Y3R > 0 ? Pat<D, P>::Y3R : 1) * Pat<D, P>::RS];   // Y3 prefix rows of the part
    float y2s[D];                   // 2 y2 prefix
    float x1[SL];                   // x1 prefix
    f4 fpart[Pat<D, P>::NW][C / 16][64];   // partial F^T of the waves
    float gin[C];                   // in-chunk row sums
    float gint[Pat<D, P>::NGI][C];  // partial q^T(Y3 q^ + 2 y2) per l block and K range (p = 1: 2 q^.y2)
};

// summary of a segment: [wave][tile][lane] f4 state, the part's Y3 rows
// [Y3R][D], y2 [D], x1 [SL]
template <int D, int P>
struct Sum {
    static constexpr size_t STATE = (size_t)Pat<D, P>::NW * Pat<D, P>::NT * 64 * 4;
    static constexpr size_t Y3 = (size_t)Pat<D, P>::Y3R * D;
    static constexpr size_t FLOATS = STATE + Y3 + D + SL;
    static constexpr size_t BYTES = (FLOATS * 4 + 255) & ~(size_t)255;
};

// One workgroup: (item = (head * NSL + slice) * NPART + part, segment).
// With one part the outputs O = F / G and G go to out and g; with several,
// each part's F and G (no division) go to fpw [head][part][N][D] and
// gpw [head][part][N] for the finalize kernel.
//
// DV (the backward's dv_n = sum_{i >= n} f(s_in) dO_i / G_i, Sec. 2.5): the
// same scan over the reversed sequence (token n at N-1-n) with the roles of
// queries and keys exchanged (q <- k, k <- q and the score scale on the
// keys), values dO scaled by 1/G per token (vsc), and no denominator: the
// numerator F is the output.
template <int D, typename T, bool CAUSAL, int MODE, bool DV, int P>
__global__ __launch_bounds__((Pat<D, P>::NTH)) void scan_kernel(const T *__restrict__ q, const T *__restrict__ k,
                                                   const T *__restrict__ v, T *__restrict__ out,
                                                   float *__restrict__ g, float *__restrict__ sums,
                                                   float *__restrict__ fpw, float *__restrict__ gpw,
                                                   const float *__restrict__ vsc, int N, int nseg,
                                                   float qs, float ks)
{
    constexpr bool DEN = !DV;   // the denominator G (forward only)
    using PT = Pat<D, P>;
    using SM = Sum<D, P>;
    constexpr int NU = PT::NU, NCH = PT::NCH, NT = PT::NT, RS = PT::RS, TS = PT::TS;
    constexpr int NPART = PT::NPART, NGW = PT::NGW, NLB = PT::NLB, Y3R = PT::Y3R;
    constexpr int NW = PT::NW, NTH = PT::NTH, LPT = PT::LPT, VPL = PT::VPL;
    constexpr int NSL = D / SL;
    constexpr int NCQ = P == 2 ? NCH : 0;   // channels with quadratic tiles
    __shared__ Smem<D, P> sm;

    const int item = blockIdx.x / nseg, seg = blockIdx.x % nseg;
    const int pp = NPART == 1 ? 0 : item % NPART;
    const int head = item / (NSL * NPART), sl = (item / NPART) % NSL;
    const int LB0 = pp * NLB;   // first Y3 row block of the part
    const int nch = (N + C - 1) / C;
    const int cbeg = (int)((long long)seg * nch / nseg), cend = (int)((long long)(seg + 1) * nch / nseg);
    const size_t hb = (size_t)head * N * D;
    q += hb;
    k += hb;
    v += hb;
    out += hb;
    if (g) g += (size_t)head * N;
    if (DV) vsc += (size_t)head * N;
    if (NPART > 1) {
        fpw += (size_t)(head * NPART + pp) * N * D;
        gpw += (size_t)(head * NPART + pp) * N;
    }
    float *sum = sums ? sums + (size_t)(item * nseg + seg) * (SM::BYTES / 4) : nullptr;

    const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, r16 = lane & 15, h = lane >> 4;
    const int gw = pp * NW + w;   // wave index over the parts
    // waves holding a Y3 row block (and K range kq) for the denominator:
    // the last NLB, or all of them with KQ per block
    constexpr int KQ = PT::KQ;
    const int lbl = KQ > 1 ? w / KQ : w - (NW - NLB), lb = LB0 + lbl;
    const int kq = KQ > 1 ? w % KQ : 0, gslot = KQ > 1 ? w : lbl;

    // ---- state, prefix sums and Y3 -------------------------------------
    f4 S[NT];
    const bool loaded = MODE == QUERY || (MODE == SCAN && seg > 0);
#pragma unroll
    for (int t = 0; t < NT; ++t)
        S[t] = loaded ? *(const f4 *)(sum + ((size_t)(w * NT + t) * 64 + lane) * 4) : f4{0.f, 0.f, 0.f, 0.f};
    // thread tid < D keeps y2[tid], D <= tid < D + SL keeps x1[tid - D]
    // (one register for both roles: the sums lie side by side after Y3)
    float colsum = 0.f;
    {
        const float *sy3 = loaded ? sum + SM::STATE : nullptr;
        constexpr int Y3N = Y3R * D;
        for (int e = tid; e < Y3N; e += NTH) sm.y3[(e / D) * RS + e % D] = loaded ? sy3[e] : 0.f;
        if (tid < D + SL) colsum = loaded ? sy3[Y3N + tid] : 0.f;
        if (tid < D) sm.y2s[tid] = 2.0f * colsum;
        else if (tid < D + SL) sm.x1[tid - D] = colsum;
    }
    // Y3 accumulator tiles of this wave, tile index yi = w + 4 kk: one part
    // takes the pairs (u, u2), u <= u2, in row order; with several parts,
    // part pp takes rows u = LB0 .. LB0 + NLB - 1, every u2
    constexpr int NYW = PT::NY3 > 0 ? (PT::NY3 + NW - 1) / NW : 1;
    f4 Y[NYW];
    int yu[NYW], yu2[NYW];
#pragma unroll
    for (int kk = 0; kk < NYW; ++kk) {
        const int yi = w + NW * kk;
        if (NPART == 1) {
            int u = 0, rem = yi;
            while (u < NU && rem >= NU - u) {
                rem -= NU - u;
                ++u;
            }
            yu[kk] = u;
            yu2[kk] = u + rem;
        } else {
            yu[kk] = LB0 + yi / NU;
            yu2[kk] = yi % NU;
        }
        Y[kk] = f4{0.f, 0.f, 0.f, 0.f};
    }
    __syncthreads();
    if (loaded) {
#pragma unroll
        for (int kk = 0; kk < NYW; ++kk) {
            if (w + NW * kk >= PT::NY3) break;
#pragma unroll
            for (int i = 0; i < 4; ++i)
                Y[kk][i] = sm.y3[(16 * (yu[kk] - LB0) + 4 * h + i) * RS + 16 * yu2[kk] + r16];
        }
    }

    // ---- staging: token tg = tid / LPT, channels LPT-way split, VPL v columns
    const int tg = tid / LPT, part = tid % LPT;
    constexpr int DP = PT::DP;
    // the next chunk's rows are loaded into registers while the current one
    // is processed (raw, converted when staged)
    RawRow<T, DP> rq, rk;
    RawRow<T, VPL> rv;
    float rvm = 1.0f;
    bool pvalid = false;
    auto prefetch = [&](int c) {
        const int n0 = c * C + tg;
        pvalid = n0 < N;
        const int n = DV ? N - 1 - n0 : n0;   // the token's place in memory
        rq.load(q + (size_t)n * D + part * DP, pvalid);
        rk.load(k + (size_t)n * D + part * DP, pvalid);
        rv.load(v + (size_t)n * D + SL * sl + VPL * part, pvalid);
        if (DV) {
            rvm = 1.0f;
            if (pvalid) rvm = vsc[n];
        }
    };
    auto stage = [&]() {
        float pq[DP], pk[DP];
#pragma unroll
        for (int i = 0; i < DP; ++i) {
            pq[i] = rq.get(i);
            pk[i] = rk.get(i);
        }
        standardise_part<D>(pq, pvalid, qs);
        standardise_part<D>(pk, pvalid, ks);
#pragma unroll
        for (int i = 0; i < DP; ++i) {
            const int ch = part * DP + i;
            sm.qrow[tg * RS + ch] = pq[i];
            sm.krow[tg * RS + ch] = pk[i];
            sm.kT[ch * TS + tg] = pk[i];
        }
#pragma unroll
        for (int i = 0; i < VPL; ++i) sm.vrow[tg * SL + VPL * part + i] = DV ? rv.get(i) * rvm : rv.get(i);
    };

    // one chunk in mode M (DELTA: state update only; QUERY: outputs only;
    // SCAN: outputs, then the update unless the segment ends here)
    auto chunk = [&](auto mc, auto ghc, int c) {
        constexpr int M = decltype(mc)::value;
        constexpr int GH = decltype(ghc)::value;   // wave class (channel blocks)
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
                    if (gw < NU) {
                        const float *qw = qr + 16 * gw + 4 * h;
    #pragma unroll
                        for (int i = 0; i < 4; ++i) F = mma(S[0][i], qw[i], F);
                    }
                    static_for<0, NCQ>([&](auto ci) {
                        constexpr int cc = decltype(ci)::value;
                        constexpr int u0 = PT::u0(cc, GH);
                        // sum over l of S[(m, l)] q_l first (the diagonal tile, holding
                        // both (m, l) and (l, m), apart at half weight), then times
                        // q_m: one multiply per channel instead of one per MFMA
                        const float qm = qr[PT::chan(cc, GH, gw)];
                        f4 Fd = {0.f, 0.f, 0.f, 0.f}, Fo = {0.f, 0.f, 0.f, 0.f};
                        static_for<u0, NU>([&](auto ui) {
                            constexpr int u = decltype(ui)::value;
                            constexpr int t = PT::first(cc, GH) + u - u0;
    #pragma unroll
                            for (int i = 0; i < 4; ++i) {
                                if constexpr (u == u0) Fd = mma(S[t][i], ql[u][i], Fd);
                                else Fo = mma(S[t][i], ql[u][i], Fo);
                            }
                        });
    #pragma unroll
                        for (int i = 0; i < 4; ++i) F[i] = fmaf(qm, fmaf(0.5f, Fd[i], Fo[i]), F[i]);
                    });
                    if constexpr (M == SCAN && CAUSAL) {
                        // in-chunk blocks of row tile rt (wave rt): the key tiles
                        // st <= rt that this part owns
                        if (w == rt) {
                            float gsum = 0.f;
    #pragma unroll
                            for (int st = 0; st <= rt; ++st) {
                                if (inchunk_owner<NPART>(rt, st) != pp) continue;
                                f4 Sc = {0.f, 0.f, 0.f, 0.f};
                                const float *kr = sm.krow + (16 * st + r16) * RS;
                                // K step kk takes channel (D/4) h + kk on lane h (both operands
                                // alike): a lane's channels are contiguous, read a few per access
    #pragma unroll
                                for (int kk = 0; kk < D / 4; ++kk) Sc = mma(kr[(D / 4) * h + kk], qr[(D / 4) * h + kk], Sc);
                                // lane: query tok, keys 16 st + 4h + i
    #pragma unroll
                                for (int i = 0; i < 4; ++i) {
                                    float wv = P == 2 ? fmaf(0.5f * Sc[i], Sc[i], 1.0f + Sc[i]) : 1.0f + Sc[i];
                                    if (st == rt && 4 * h + i > r16) wv = 0.0f;
                                    Sc[i] = wv;
                                    gsum += wv;
                                }
    #pragma unroll
                                for (int i = 0; i < 4; ++i)
                                    F = mma(sm.vrow[(16 * st + 4 * h + i) * SL + r16], Sc[i], F);
                            }
                            if (DEN) {
                                gsum = rows4_sum(gsum);
                                if (h == 0) sm.gin[tok] = gsum;
                            }
                        }
                    }
                    sm.fpart[w][rt][lane] = F;
                    // denominator: q^T (Y3 q + 2 y2) over l block lb (p = 1: 2 q.y2),
                    // K steps kq KK .. kq KK + KK - 1 of the contraction
                    if (DEN && lbl >= 0) {
                        constexpr int KK = D / 4 / KQ;
                        f4 Tq;
    #pragma unroll
                        for (int i = 0; i < 4; ++i) Tq[i] = kq == 0 ? sm.y2s[16 * lb + 4 * h + i] : 0.f;
                        if constexpr (P == 2) {
                            const float *yr = sm.y3 + (16 * lbl + r16) * RS + 4 * KK * kq + h;
                            const float *qk = qr + 4 * KK * kq + h;
    #pragma unroll
                            for (int kk = 0; kk < KK; ++kk) Tq = mma(yr[4 * kk], qk[4 * kk], Tq);
                        }
                        float gq = 0.f;
    #pragma unroll
                        for (int i = 0; i < 4; ++i) gq = fmaf(qr[16 * lb + 4 * h + i], Tq[i], gq);
                        gq = rows4_sum(gq);
                        if (h == 0) sm.gint[gslot][tok] = gq;
                    }
                }
                __syncthreads();
                // ---- outputs O = F / G: token tg, columns VPL part .. + VPL - 1
                // (part 0 of several adds the count and x1; each part its
                // share of the rest)
                {
                    const int n = n0 + tg;
                    if (n < N) {
                        const int nm = DV ? N - 1 - n : n;   // the token's place in memory
                        const int rt = tg >> 4, t16 = tg & 15;
                        float G = 1.f;
                        if (DEN) {
                            float gsum = 0.f;
    #pragma unroll
                            for (int ww = 0; ww < PT::NGI; ++ww) gsum += sm.gint[ww][tg];
                            G = (pp == 0 ? (M == QUERY ? (float)N : (float)n0) : 0.f) + 0.5f * gsum;
                            if (M == SCAN && CAUSAL) G += sm.gin[tg];
                        }
                        const float rG = 1.0f / G;
    #pragma unroll
                        for (int i = 0; i < VPL; ++i) {
                            const int j = VPL * part + i;
                            float F = pp == 0 ? sm.x1[j] : 0.f;
    #pragma unroll
                            for (int ww = 0; ww < NW; ++ww) F += sm.fpart[ww][rt][16 * (j >> 2) + t16][j & 3];
                            if (NPART == 1) io<T>::st(out, (size_t)nm * D + SL * sl + j, DEN ? F * rG : F);
                            else fpw[(size_t)nm * D + SL * sl + j] = F;
                        }
                        if (DEN) {
                            if (NPART == 1) {
                                if (g && sl == 0 && part == 0) g[n] = G;
                            } else if (sl == 0 && part == 0) {
                                gpw[n] = G;
                            }
                        }
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
                if (gw < NU) {
                    const float *kl = sm.kT + (16 * gw + r16) * TS + h;
    #pragma unroll
                    for (int ks = 0; ks < C / 4; ++ks) S[0] = mma(kl[4 * ks], Vb[ks], S[0]);
                }
                static_for<0, NCQ>([&](auto ci) {
                    constexpr int cc = decltype(ci)::value;
                    constexpr int u0 = PT::u0(cc, GH);
                    const float *km = sm.kT + PT::chan(cc, GH, gw) * TS + h;
                    float Bm[C / 4];
    #pragma unroll
                    for (int ks = 0; ks < C / 4; ++ks) Bm[ks] = km[4 * ks] * Vb[ks];
                    static_for<u0, NU>([&](auto ui) {
                        constexpr int u = decltype(ui)::value;
                        constexpr int t = PT::first(cc, GH) + u - u0;
    #pragma unroll
                        for (int ks = 0; ks < C / 4; ++ks) S[t] = mma(Ak[u][ks], Bm[ks], S[t]);
                    });
                });
    #pragma unroll
                for (int kk = 0; kk < NYW; ++kk) {
                    if (!DEN || w + NW * kk >= PT::NY3) break;
                    const float *a = sm.kT + (16 * yu[kk] + r16) * TS + h;
                    const float *b = sm.kT + (16 * yu2[kk] + r16) * TS + h;
    #pragma unroll
                    for (int ks = 0; ks < C / 4; ++ks) Y[kk] = mma(a[4 * ks], b[4 * ks], Y[kk]);
                }
                if (tid < D) {
                    if (DEN) {
                        float s = 0.f;
    #pragma unroll 8
                        for (int t = 0; t < C; ++t) s += sm.krow[t * RS + tid];
                        colsum += s;
                    }
                } else if (tid < D + SL) {
                    float s = 0.f;
    #pragma unroll 8
                    for (int t = 0; t < C; ++t) s += sm.vrow[t * SL + tid - D];
                    colsum += s;
                }
                __syncthreads();
                // the prefix after this chunk, for the next chunk's outputs
    #pragma unroll
                for (int kk = 0; kk < NYW; ++kk) {
                    if (!DEN || w + NW * kk >= PT::NY3) break;
    #pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int l = 16 * yu[kk] + 4 * h + i, m = 16 * yu2[kk] + r16;
                        sm.y3[(l - 16 * LB0) * RS + m] = Y[kk][i];
                        if (NPART == 1) sm.y3[m * RS + l] = Y[kk][i];
                    }
                }
                if (tid < D) sm.y2s[tid] = 2.0f * colsum;
                else if (tid < D + SL) sm.x1[tid - D] = colsum;
            }
            __syncthreads();
    };
    with_wave_class<D, P>(gw, [&](auto ghc) {
        if constexpr (MODE == BOTH) {
            // non-causal, one segment: the totals first, then every query
            prefetch(cbeg);
            for (int c = cbeg; c < cend; ++c) chunk(std::integral_constant<int, DELTA>{}, ghc, c);
            prefetch(cbeg);
            for (int c = cbeg; c < cend; ++c) chunk(std::integral_constant<int, QUERY>{}, ghc, c);
        } else {
            prefetch(cbeg);
            for (int c = cbeg; c < cend; ++c) chunk(std::integral_constant<int, MODE>{}, ghc, c);
        }
    });

    if constexpr (MODE == DELTA) {
        // this segment's sums: state, Y3 (from LDS, written by the last
        // update), y2, x1
#pragma unroll
        for (int t = 0; t < NT; ++t) *(f4 *)(sum + ((size_t)(w * NT + t) * 64 + lane) * 4) = S[t];
        float *sy3 = sum + SM::STATE;
        constexpr int Y3N = Y3R * D;
        for (int e = tid; e < Y3N; e += NTH) sy3[e] = sm.y3[(e / D) * RS + e % D];
        if (tid < D + SL) sy3[Y3N + tid] = colsum;
    }
}

// Several parts: out = (sum of the parts' F) / (sum of their G), g = that
// sum; 16 tokens per workgroup, 16 threads per token, D/16 columns each.
template <int D, int P, typename T, bool DIV>
__global__ __launch_bounds__(256) void finalize_kernel(const float *__restrict__ fpw,
                                                       const float *__restrict__ gpw,
                                                       T *__restrict__ out, float *__restrict__ g,
                                                       int N, int nblk)
{
    constexpr int NP = Pat<D, P>::NPART, CPT = D / 16;
    static_assert(CPT % 4 == 0, "float4 columns");
    const int head = blockIdx.x / nblk, n = (blockIdx.x % nblk) * 16 + (threadIdx.x >> 4);
    const int cg = threadIdx.x & 15;
    if (n >= N) return;
    float G = 0.f;   // (no division: the sum of F alone)
    f4 F[CPT / 4];
#pragma unroll
    for (int i = 0; i < CPT / 4; ++i) F[i] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int pp = 0; pp < NP; ++pp) {
        const size_t row = (size_t)(head * NP + pp) * N + n;
        if (DIV) G += gpw[row];
        const f4 *src = (const f4 *)(fpw + row * D + CPT * cg);
#pragma unroll
        for (int i = 0; i < CPT / 4; ++i) F[i] += src[i];
    }
    const float rG = DIV ? 1.0f / G : 1.0f;
    const size_t o = ((size_t)head * N + n) * D + CPT * cg;
#pragma unroll
    for (int i = 0; i < CPT; ++i) io<T>::st(out, o + i, F[i / 4][i % 4] * rG);
    if (DIV && g && cg == 0) g[(size_t)head * N + n] = G;
}

// Workspace: segment sums (several segments), then the parts' F and G
// (several parts).
template <int D, int P>
struct Plan {
    int items, nch, nseg;
    size_t sum_bytes, fp_bytes, gp_bytes;
    Plan(int BH, int N)
    {
        constexpr int NP = Pat<D, P>::NPART;
        items = BH * (D / SL) * NP;
        nch = (N + C - 1) / C;
        // D <= 32: under 128 VGPRs, so two workgroups share a CU
        nseg = nseg_of(items, nch, D <= 32 ? 2 * TARGET_BLOCKS : TARGET_BLOCKS);
        sum_bytes = nseg > 1 ? a256((size_t)items * nseg * Sum<D, P>::BYTES) : 0;
        fp_bytes = NP > 1 ? a256((size_t)BH * NP * N * D * 4) : 0;
        gp_bytes = NP > 1 ? a256((size_t)BH * NP * N * 4) : 0;
    }
    size_t bytes() const { return sum_bytes + fp_bytes + gp_bytes; }
};

// The forward (DV = false: O = F / G and G) or the backward's dv (DV = true:
// q <- k, k <- q, v <- dout scaled by vsc = 1/G, the score scale on the keys).
template <int D, typename T, bool DV, int P>
hipError_t launch(const void *q, const void *k, const void *v, const float *vsc, void *out,
                  float *g, int BH, int N, int causal, float qs, float ks, void *ws, hipStream_t st)
{
    using PT = Pat<D, P>;
    using SM = Sum<D, P>;
    const Plan<D, P> pl(BH, N);
    const int items = pl.items, nseg = pl.nseg;
    const int nblk = (N + 15) / 16;   // finalize: 16 rows per workgroup
    if (!f32mfma_fwd_grids_fit(BH, N, D, P)) return hipErrorInvalidConfiguration;
    const dim3 grid((unsigned)(items * nseg)), blk(PT::NTH);
    const T *Q = (const T *)q, *K = (const T *)k, *V = (const T *)v;
    T *O = (T *)out;
    float *sums = nseg > 1 ? (float *)ws : nullptr;
    float *fpw = pl.fp_bytes ? (float *)((char *)ws + pl.sum_bytes) : nullptr;
    float *gpw = pl.gp_bytes ? (float *)((char *)ws + pl.sum_bytes + pl.fp_bytes) : nullptr;
    const size_t stride = SM::BYTES / 4;
    const dim3 pgrid((unsigned)((SM::FLOATS + 255) / 256), items);
    if (causal) {
        if (nseg > 1) {
            hipLaunchKernelGGL((scan_kernel<D, T, true, DELTA, DV, P>), grid, blk, 0, st, Q, K, V,
                               O, g, sums, fpw, gpw, vsc, N, nseg, qs, ks);
            hipLaunchKernelGGL(prefix_kernel, pgrid, dim3(256), 0, st, sums, nseg, SM::FLOATS,
                               stride, 1);
        }
        hipLaunchKernelGGL((scan_kernel<D, T, true, SCAN, DV, P>), grid, blk, 0, st, Q, K, V, O, g,
                           sums, fpw, gpw, vsc, N, nseg, qs, ks);
    } else if (nseg == 1) {
        hipLaunchKernelGGL((scan_kernel<D, T, false, BOTH, DV, P>), grid, blk, 0, st, Q, K, V, O,
                           g, nullptr, fpw, gpw, vsc, N, nseg, qs, ks);
    } else {
        hipLaunchKernelGGL((scan_kernel<D, T, false, DELTA, DV, P>), grid, blk, 0, st, Q, K, V, O,
                           g, sums, fpw, gpw, vsc, N, nseg, qs, ks);
        hipLaunchKernelGGL(prefix_kernel, pgrid, dim3(256), 0, st, sums, nseg, SM::FLOATS, stride,
                           0);
        hipLaunchKernelGGL((scan_kernel<D, T, false, QUERY, DV, P>), grid, blk, 0, st, Q, K, V, O,
                           g, sums, fpw, gpw, vsc, N, nseg, qs, ks);
    }
    if constexpr (PT::NPART > 1) {
        hipLaunchKernelGGL((finalize_kernel<D, P, T, !DV>), dim3((unsigned)(BH * nblk)), dim3(256),
                           0, st, fpw, gpw, O, g, N, nblk);
    }
    return hipGetLastError();
}

template <bool DV, typename T, int P>
hipError_t launch_dt(const void *q, const void *k, const void *v, const float *vsc, void *out,
                     float *g, int BH, int N, int D, int causal, float qs, float ks, void *ws,
                     hipStream_t st)
{
    switch (D) {
    case 16: return launch<16, T, DV, P>(q, k, v, vsc, out, g, BH, N, causal, qs, ks, ws, st);
    case 32: return launch<32, T, DV, P>(q, k, v, vsc, out, g, BH, N, causal, qs, ks, ws, st);
    case 64: return launch<64, T, DV, P>(q, k, v, vsc, out, g, BH, N, causal, qs, ks, ws, st);
    case 128: return launch<128, T, DV, P>(q, k, v, vsc, out, g, BH, N, causal, qs, ks, ws, st);
    }
    return hipErrorInvalidValue;
}

template <bool DV>
hipError_t launch_d(const void *q, const void *k, const void *v, const float *vsc, void *out,
                    float *g, int BH, int N, int D, int p, int causal, int is_bf16, float qs,
                    float ks, void *ws, hipStream_t st)
{
    if (!f32mfma_applies(D, p, is_bf16)) return hipErrorInvalidValue;
    if (is_bf16)
        return p == 2 ? launch_dt<DV, bf16_t, 2>(q, k, v, vsc, out, g, BH, N, D, causal, qs, ks, ws, st)
                      : launch_dt<DV, bf16_t, 1>(q, k, v, vsc, out, g, BH, N, D, causal, qs, ks, ws, st);
    return p == 2 ? launch_dt<DV, float, 2>(q, k, v, vsc, out, g, BH, N, D, causal, qs, ks, ws, st)
                  : launch_dt<DV, float, 1>(q, k, v, vsc, out, g, BH, N, D, causal, qs, ks, ws, st);
}

}  // namespace m32

bool f32mfma_applies(int D, int p, int is_bf16)
{
    (void)is_bf16;   // every dtype (bf16 D = 64, p = 2 only where the fp16 kernels do not serve)
    return (p == 1 || p == 2) && (D == 16 || D == 32 || D == 64 || D == 128);
}

namespace m32 {
template <int D, int P>
bool grids_fit(int BH, int N)
{
    const Plan<D, P> pl(BH, N);
    return grid_fits((long long)pl.items * pl.nseg, Pat<D, P>::NTH) &&
           (Pat<D, P>::NPART == 1 || grid_fits((long long)BH * ((N + 15) / 16), 256));
}
}  // namespace m32

bool f32mfma_fwd_grids_fit(int BH, int N, int D, int p)
{
    using namespace m32;
    switch (D) {
    case 16: return p == 1 ? grids_fit<16, 1>(BH, N) : grids_fit<16, 2>(BH, N);
    case 32: return p == 1 ? grids_fit<32, 1>(BH, N) : grids_fit<32, 2>(BH, N);
    case 64: return p == 1 ? grids_fit<64, 1>(BH, N) : grids_fit<64, 2>(BH, N);
    case 128: return p == 1 ? grids_fit<128, 1>(BH, N) : grids_fit<128, 2>(BH, N);
    }
    return false;
}

size_t f32mfma_fwd_workspace(int BH, int N, int D, int p)
{
    using namespace m32;
    if (p == 1) {
        switch (D) {
        case 16: return Plan<16, 1>(BH, N).bytes();
        case 32: return Plan<32, 1>(BH, N).bytes();
        case 64: return Plan<64, 1>(BH, N).bytes();
        case 128: return Plan<128, 1>(BH, N).bytes();
        }
        return 0;
    }
    switch (D) {
    case 16: return Plan<16, 2>(BH, N).bytes();
    case 32: return Plan<32, 2>(BH, N).bytes();
    case 64: return Plan<64, 2>(BH, N).bytes();
    case 128: return Plan<128, 2>(BH, N).bytes();
    }
    return 0;
}

hipError_t f32mfma_fwd(const void *q, const void *k, const void *v, void *out, float *g, int BH,
                       int N, int D, int p, int causal, int is_bf16, float qs, void *ws,
                       hipStream_t st)
{
    return m32::launch_d<false>(q, k, v, nullptr, out, g, BH, N, D, p, causal, is_bf16, qs, 1.0f,
                                ws, st);
}

hipError_t f32mfma_dv(const void *q, const void *k, const void *dout, const float *rg, void *dv,
                      int BH, int N, int D, int p, int causal, int is_bf16, float qs, void *ws,
                      hipStream_t st)
{
    return m32::launch_d<true>(k, q, dout, rg, dv, nullptr, BH, N, D, p, causal, is_bf16, 1.0f,
                               qs, ws, st);
}

}  // namespace fm

// Fastmax backward on float32 MFMA (v_mfma_f32_16x16x4_f32), p = 1 and 2, the
// cases of the float32 MFMA forward (p = 1: f' = 1, the linear tiles only).  Sec. 2.5's custom gradient: only O and G are
// kept from the forward, q^ and k^ are recomputed, and the moments are
// rebuilt by scans instead of stored.  With u_i = dO_i / G_i,
// c_i = (dO_i . O_i) / G_i and s_in = q~_i . k^_n (q~ = tau q^):
//
//   dv_n  = sum_{i >= n} f(s_in) u_i
//   dq~_i = sum_{n <= i} f'(s_in) (u_i . v_n - c_i) k^_n
//   dk^_n = sum_{i >= n} f'(s_in) (u_i . v_n - c_i) q~_i       (f' = 1 + s)
//
// (all n, i for the non-causal problem), then back through the
// standardisation (Eqs. 6-7).  dv is the forward's scan over the reversed
// sequence with queries and keys exchanged (fm_f32_mfma.hip).  dq~ and dk^
// are one "gradient scan" run twice with the roles exchanged: with state
// keys X, state values VS, state weights w, contraction features Z,
// contraction columns UC and contraction scalars z,
//
//   out_t = sum_{r before t} f'(Z_t . X_r) (UC_t . VS_r + z_t w_r) X_r
//
// dq~: X = k^, VS = v, w = 1, Z = q~, UC = u, z = -c (forward order);
// dk^: X = q~, VS = u, w = c, Z = k^, UC = v, z = -1 (reverse order).
// Expanded, out_t[l] = sum_c UC_tc L[l][c] + z_t y2w[l]
//                      + sum_m Z_tm (sum_c UC_tc Q[m,l][c] + z_t Y3w[m][l])
// with the moment state L = sum_r X_r VS_r^T, Q[m,l] = sum_r X_rm X_rl VS_r^T
// (the forward's state, per 16-column slice of VS), y2w = sum_r w_r X_r and
// Y3w = sum_r w_r X_r X_r^T; chunks of 32 tokens add their in-chunk pairs
// directly.
//
// The state tiles are kept transposed with respect to the forward's: lane
// (r16, h) element i holds feature 16u + r16, column 4h + i, so element i
// is the A operand of K step i of a contraction over the columns, whose B
// operand UC_t[4h + i] is shared by every tile; each tile gives
// T[l][t] = sum_c Q[m,l][c] UC_tc in the layout (token r16, feature 4h + i)
// of the per-wave output rows.  A diagonal tile (both orders of its pairs)
// adds Z_tm T[l] to out_t[l]; an off-diagonal tile (m's block below l's)
// also adds sum_l Z_tl T[l] to out_t[m].  Each wave folds all its terms for
// one 16-feature block into registers and stores the block once into its own
// LDS region (LDS float atomics, measured, cost more than the MFMAs); the
// chunk's rows, summed over the eight regions, are added to the float32
// gradient with global float atomics (the column slices and feature parts of
// a head add into the same rows).
#include <hip/hip_runtime.h>

#include <limits.h>

#include "fm_common.h"
#include "fm_f32_mfma.h"
#include "fm_internal.h"

namespace fm {
namespace m32 {

// Tokens of the per-wave output blocks: the whole chunk where the waves'
// blocks fit 64 KB of LDS, else one 16-token row tile at a time.
template <int D, int P>
constexpr int out_tokens() { return Pat<D, P>::NW * D * (C + 4) * 4 <= 65536 ? C : 16; }

template <int D, int P>
struct alignas(16) GSmem {
    float xrow[C * Pat<D, P>::RS];  // state keys X [token][channel]
    float xT[D * Pat<D, P>::TS];    // X [channel][token]
    alignas(16) float zrow[C * (D + 4)];   // contraction features Z [token][channel] (16-byte rows)
    float vs[C * SL];              // state values, this slice [token][column]
    float uc[C * SL];              // contraction columns, this slice
    float wt[C];                   // state weights w
    float zt[C];                   // contraction scalars z
    float y3[(P == 2 ? 16 : 1) * Pat<D, P>::RS];   // the item's row block of Y3w (p = 2)
    float y2[P == 2 ? 16 : D];     // its entries of y2w (p = 1: all of y2w)
    alignas(16) float ob[Pat<D, P>::NW][D * (out_tokens<D, P>() + 4)];   // each wave's outputs [feature][token]
};

// Segment summary: [wave][tile][lane] f4 state, the Y3w row block [16][D]
// and y2w [16] (p = 1: y2w [D]).
template <int D, int P>
struct GSum {
    static constexpr size_t STATE = (size_t)Pat<D, P>::NW * Pat<D, P>::NT * 64 * 4;
    static constexpr int Y3N = P == 2 ? 16 * D : 0, Y2N = P == 2 ? 16 : D;
    static constexpr size_t FLOATS = STATE + Y3N + Y2N;
    static constexpr size_t BYTES = (FLOATS * 4 + 255) & ~(size_t)255;
};

// One workgroup: (item = (head * NSL + slice) * NPART + part, segment).  The
// item (slice, part) with index sl * NPART + part = b < D/16 also keeps row
// block b of Y3w and y2w (p = 1: item 0 keeps y2w); slice 0 adds the z_t w_r
// term of the in-chunk pairs.  p = 1 (f' = 1): only the linear tiles, no
// Y3w, in-chunk weights UC_t.VS_r + z_t w_r.
template <int D, typename T, bool CAUSAL, int MODE, bool REV, int P>
__global__ __launch_bounds__((Pat<D, P>::NTH)) void grad_kernel(
    const T *__restrict__ X, const T *__restrict__ Z, const T *__restrict__ VS,
    const T *__restrict__ UC, const float *__restrict__ vsm, const float *__restrict__ ucm,
    const float *__restrict__ wv, const float *__restrict__ zv, float *__restrict__ outh,
    float *__restrict__ sums, int N, int nseg, float xs, float zsc)
{
    using PT = Pat<D, P>;
    using GS = GSum<D, P>;
    constexpr int NU = PT::NU, NCH = PT::NCH, NT = PT::NT, RS = PT::RS, TS = PT::TS;
    constexpr int NPART = PT::NPART, NGW = PT::NGW;
    constexpr int NW = PT::NW, NTH = PT::NTH, LPT = PT::LPT, VPL = PT::VPL;
    constexpr int NSL = D / SL;
    constexpr int ZS = D + 4;   // row stride of Z
    // output block: FT tokens; its feature stride puts the lanes (token r16,
    // features 4h + i) of one LDS store in 64 distinct banks
    constexpr int FT = out_tokens<D, P>(), OS = FT + 4;
    constexpr int NCQ = P == 2 ? NCH : 0;   // channels with quadratic tiles
    __shared__ GSmem<D, P> sm;

    const int item = blockIdx.x / nseg, seg = blockIdx.x % nseg;
    const int pp = NPART == 1 ? 0 : item % NPART;
    const int head = item / (NSL * NPART), sl = (item / NPART) % NSL;
    const int yb = item % (NSL * NPART);
    // the item's Y3w row block, if any (p = 1: 0 for the item that keeps y2w)
    const int ylb = (P == 2 ? yb < NU : yb == 0) ? yb : -1;
    const bool scal = sl == 0;
    const int nch = (N + C - 1) / C;
    const int cbeg = (int)((long long)seg * nch / nseg), cend = (int)((long long)(seg + 1) * nch / nseg);
    const size_t hb = (size_t)head * N * D;
    X += hb;
    Z += hb;
    VS += hb;
    UC += hb;
    outh += hb;
    if (vsm) vsm += (size_t)head * N;
    if (ucm) ucm += (size_t)head * N;
    if (wv) wv += (size_t)head * N;
    if (zv) zv += (size_t)head * N;
    float *sum = sums ? sums + (size_t)(item * nseg + seg) * (GS::BYTES / 4) : nullptr;

    const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, r16 = lane & 15, h = lane >> 4;
    const int gw = pp * NW + w;

    // ---- state, Y3w block, y2w -----------------------------------------
    f4 S[NT];
    const bool loaded = MODE == QUERY || (MODE == SCAN && seg > 0);
#pragma unroll
    for (int t = 0; t < NT; ++t)
        S[t] = loaded ? *(const f4 *)(sum + ((size_t)(w * NT + t) * 64 + lane) * 4) : f4{0.f, 0.f, 0.f, 0.f};
    // thread tid < Y2N of an item with a Y3w block: y2w[16 ylb + tid] (p = 1: y2w[tid])
    float y2reg = 0.f;
    {
        const float *sy = loaded ? sum + GS::STATE : nullptr;
        for (int e = tid; e < GS::Y3N; e += NTH) sm.y3[(e / D) * RS + e % D] = loaded ? sy[e] : 0.f;
        if (tid < GS::Y2N) {
            y2reg = loaded ? sy[GS::Y3N + tid] : 0.f;
            sm.y2[tid] = y2reg;
        }
    }
    // Y3w tiles (ylb, u2), u2 = w + 4 kk
    constexpr int NYW = (NU + NW - 1) / NW;
    f4 Y[NYW];
#pragma unroll
    for (int kk = 0; kk < NYW; ++kk) Y[kk] = f4{0.f, 0.f, 0.f, 0.f};
    __syncthreads();
    if (P == 2 && loaded && ylb >= 0) {
#pragma unroll
        for (int kk = 0; kk < NYW; ++kk) {
            const int u2 = w + NW * kk;
            if (u2 >= NU) break;
#pragma unroll
            for (int i = 0; i < 4; ++i) Y[kk][i] = sm.y3[(4 * h + i) * RS + 16 * u2 + r16];
        }
    }

    // ---- staging: token tg = tid / 8, channels 8-way split, 2 columns ---
    const int tg = tid / LPT, part = tid % LPT;
    constexpr int DP = PT::DP;
    // the next chunk's rows, raw (converted when staged, so that the loads
    // overlap the current chunk)
    RawRow<T, DP> rx, rz;
    RawRow<T, VPL> rvs, ruc;
    float rvm = 1.f, rum = 1.f, pw = 0.f, pzv = 0.f;
    bool pvalid = false;
    auto prefetch = [&](int c) {
        const int n0 = c * C + tg;
        pvalid = n0 < N;
        const int n = REV ? N - 1 - n0 : n0;   // the token's place in memory
        rx.load(X + (size_t)n * D + part * DP, pvalid);
        rz.load(Z + (size_t)n * D + part * DP, pvalid);
        const size_t e = (size_t)n * D + SL * sl + VPL * part;
        rvs.load(VS + e, pvalid);
        ruc.load(UC + e, pvalid);
        rvm = 1.f;
        rum = 1.f;
        pw = pvalid ? 1.f : 0.f;
        pzv = pvalid ? 1.f : 0.f;
        if (pvalid) {
            if (vsm) rvm = vsm[n];
            if (ucm) rum = ucm[n];
            if (wv) pw = wv[n];
            if (zv) pzv = zv[n];
        }
    };
    auto stage = [&]() {
        float px[DP], pz[DP];
#pragma unroll
        for (int i = 0; i < DP; ++i) {
            px[i] = rx.get(i);
            pz[i] = rz.get(i);
        }
        standardise_part<D>(px, pvalid, xs);
        standardise_part<D>(pz, pvalid, zsc);
#pragma unroll
        for (int i = 0; i < DP; ++i) {
            const int ch = part * DP + i;
            sm.xrow[tg * RS + ch] = px[i];
            sm.xT[ch * TS + tg] = px[i];
            sm.zrow[tg * ZS + ch] = pz[i];
        }
#pragma unroll
        for (int i = 0; i < VPL; ++i) {
            sm.vs[tg * SL + VPL * part + i] = rvs.get(i) * rvm;
            sm.uc[tg * SL + VPL * part + i] = ruc.get(i) * rum;
        }
        if (part == 0) {
            sm.wt[tg] = pw;
            sm.zt[tg] = pvalid ? -pzv : 0.f;
        }
    };

    // one chunk in mode M (DELTA: state update only; QUERY: outputs only;
    // SCAN: outputs, then the update unless the segment ends here)
    auto chunk = [&](auto mc, auto ghc, int c) {
        constexpr int M = decltype(mc)::value;
        constexpr int GH = decltype(ghc)::value;   // wave class (channel blocks)
        const int n0 = c * C;
        // the waves' output blocks of tokens t0 .. t0 + FT - 1 (summed) into
        // the float32 gradient
        // (a thread takes feature d of four consecutive tokens: one 16-byte
        // LDS read per wave region, lanes 80 or 144 bytes apart, which is
        // conflict-free; consecutive lanes add to consecutive features of a row)
        auto flush = [&](int t0) {
            for (int e = tid; e < (FT / 4) * D; e += NTH) {
                const int j4 = e / D, d = e % D, o = d * OS + 4 * j4;
                f4 val = *(const f4 *)&sm.ob[0][o];
#pragma unroll
                for (int ww = 1; ww < NW; ++ww) val += *(const f4 *)&sm.ob[ww][o];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int n = n0 + t0 + 4 * j4 + j;
                    if (n < N) atomicAdd(outh + (size_t)(REV ? N - 1 - n : n) * D + d, val[j]);
                }
            }
        };
        stage();
        if (c + 1 < cend) prefetch(c + 1);
        __syncthreads();

        if constexpr (M != DELTA) {
#pragma unroll
            for (int rt = 0; rt < C / 16; ++rt) {
                const int tok = 16 * rt + r16;
                const float *zr = sm.zrow + tok * ZS;
                // this wave's outputs of the row tile, every (feature, token)
                // written once: feature f of token tok at ocol[f * OS]
                float *ocol = sm.ob[w] + (FT == C ? tok : r16);
                float ub[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) ub[i] = sm.uc[tok * SL + 4 * h + i];
                // in-chunk pairs: key tile st <= rt on wave b of the owning part;
                // the weights here, their products with X by output block below
                float Wt[2][4] = {};
                bool ich[2] = {false, false};
                if constexpr (M == SCAN && CAUSAL) {
#pragma unroll
                    for (int st = 0; st < 2; ++st) {
                        ich[st] = st <= rt && inchunk_owner<NPART>(rt, st) == pp &&
                                  w == rt * (rt + 1) / 2 + st;
                        if (!ich[st]) continue;
                        // S^T and P^T: lane (token tok, keys 16 st + 4h + i)
                        f4 Sc = {0.f, 0.f, 0.f, 0.f}, Pc = {0.f, 0.f, 0.f, 0.f};
                        if constexpr (P == 2) {
                            const float *xr = sm.xrow + (16 * st + r16) * RS;
                            // K step kk takes channel (D/4) h + kk on lane h (both operands
                            // alike): a lane's channels are contiguous, read a few per access
#pragma unroll
                            for (int kk = 0; kk < D / 4; ++kk) Sc = mma(xr[(D / 4) * h + kk], zr[(D / 4) * h + kk], Sc);
                        }
                        const float *vr = sm.vs + (16 * st + r16) * SL;
#pragma unroll
                        for (int kk = 0; kk < 4; ++kk)
                            Pc = mma(vr[4 * kk + h], sm.uc[tok * SL + 4 * kk + h], Pc);
                        const float zs = scal ? sm.zt[tok] : 0.f;
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            float wgt = fmaf(zs, sm.wt[16 * st + 4 * h + i], Pc[i]);
                            if (P == 2) wgt *= 1.0f + Sc[i];
                            if (st == rt && 4 * h + i > r16) wgt = 0.0f;
                            Wt[st][i] = wgt;
                        }
                    }
                }
                // the item's Y3w block (p = 2: its contraction split by K range over
                // the first YQ waves; p = 1: z_t y2w[l] to every block, wave NW - 1)
                constexpr int YQ = D / 4 < NW ? D / 4 : NW;
                const bool yw = ylb >= 0 && (P == 2 ? w < YQ : w == NW - 1);
                const float zst = sm.zt[tok];
                // quadratic tiles by output block u, from the last block down: tile
                // (m, u) of the wave's channel m = chan(cc) adds Z_m T[l] to out[l], l in
                // block u, and (off the diagonal) sum_l Z_l T[l] to out[m], which is
                // complete when the loop reaches m's own block u0
                float dmv[NCH];
#pragma unroll
                for (int cc = 0; cc < NCH; ++cc) dmv[cc] = 0.f;
                static_for<0, NU>([&](auto ri) {
                    constexpr int u = NU - 1 - decltype(ri)::value;
                    const f4 zlu = *(const f4 *)(zr + 16 * u + 4 * h);
                    f4 a4 = {0.f, 0.f, 0.f, 0.f};
                    static_for<0, NCQ>([&](auto ci) {
                        constexpr int cc = decltype(ci)::value;
                        constexpr int u0 = PT::u0(cc, GH);
                        if constexpr (u >= u0) {
                            constexpr int t = PT::first(cc, GH) + u - u0;
                            const float zm = zr[PT::chan(cc, GH, gw)];
                            f4 Tt = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                            for (int i = 0; i < 4; ++i) Tt = mma(S[t][i], ub[i], Tt);
#pragma unroll
                            for (int i = 0; i < 4; ++i) a4[i] = fmaf(zm, Tt[i], a4[i]);
                            if constexpr (u > u0) {
#pragma unroll
                                for (int i = 0; i < 4; ++i) dmv[cc] = fmaf(zlu[i], Tt[i], dmv[cc]);
                            }
                        }
                        if constexpr (u == u0 && u0 + 1 < NU) {
                            const float dm = rows4_sum(dmv[cc]);
                            const int ml = PT::chan(cc, GH, gw) & 15;
#pragma unroll
                            for (int i = 0; i < 4; ++i)
                                if (h == (ml >> 2) && i == (ml & 3)) a4[i] += dm;
                        }
                    });
                    if (P == 1 && yw) {
#pragma unroll
                        for (int i = 0; i < 4; ++i) a4[i] = fmaf(zst, sm.y2[16 * u + 4 * h + i], a4[i]);
                    }
                    if constexpr (M == SCAN && CAUSAL) {
#pragma unroll
                        for (int st = 0; st < 2; ++st) {
                            if (!ich[st]) continue;
                            // out[l] += sum_r W[t][r] X_r[l]
#pragma unroll
                            for (int i = 0; i < 4; ++i)
                                a4 = mma(sm.xrow[(16 * st + 4 * h + i) * RS + 16 * u + r16], Wt[st][i], a4);
                        }
                    }
#pragma unroll
                    for (int i = 0; i < 4; ++i) ocol[(16 * u + 4 * h + i) * OS] = a4[i];
                });
                // terms of a single block, added to the wave's stored block (rather
                // than selected into every block's registers):
                // the linear tile, out[l] += sum_c UC_c L[l][c] for l in block gw
                if (gw < NU) {
                    f4 Tl = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int i = 0; i < 4; ++i) Tl = mma(S[0][i], ub[i], Tl);
#pragma unroll
                    for (int i = 0; i < 4; ++i) ocol[(16 * gw + 4 * h + i) * OS] += Tl[i];
                }
                // and the Y3w block, out[l] += z_t (y2w[l] + sum_m Y3w[l][m] Z_tm)
                // for l in block ylb: wave w adds K steps w KK .. w KK + KK - 1 of
                // the sum over m (wave 0 the y2w term) to its own stored block,
                // and the flush adds the waves' blocks
                if (P == 2 && yw) {
                    constexpr int KK = D / 4 / YQ;
                    f4 Tq;
#pragma unroll
                    for (int i = 0; i < 4; ++i) Tq[i] = w == 0 ? sm.y2[4 * h + i] : 0.f;
                    const float *yr = sm.y3 + r16 * RS + 4 * KK * w + h;
                    const float *zk = zr + 4 * KK * w + h;
#pragma unroll
                    for (int kk = 0; kk < KK; ++kk) Tq = mma(yr[4 * kk], zk[4 * kk], Tq);
#pragma unroll
                    for (int i = 0; i < 4; ++i) ocol[(16 * ylb + 4 * h + i) * OS] += zst * Tq[i];
                }
                if constexpr (FT == 16) {
                    __syncthreads();
                    flush(16 * rt);
                    __syncthreads();   // the blocks are written again by the next row tile
                }
            }
            if constexpr (FT == C) {
                __syncthreads();
                flush(0);
            }
        }
        if constexpr (M != QUERY) {
            if (M == SCAN && c + 1 == cend) return;   // the next segment starts from its prefix
            // ---- state update (transposed tiles), Y3w block, y2w --------------
            float Ak[NU][C / 4], Vb[C / 4];
#pragma unroll
            for (int u = 0; u < NU; ++u)
#pragma unroll
                for (int ks = 0; ks < C / 4; ++ks) Ak[u][ks] = sm.xT[(16 * u + r16) * TS + 4 * ks + h];
#pragma unroll
            for (int ks = 0; ks < C / 4; ++ks) Vb[ks] = sm.vs[(4 * ks + h) * SL + r16];
            if (gw < NU) {
                const float *xl = sm.xT + (16 * gw + r16) * TS + h;
#pragma unroll
                for (int ks = 0; ks < C / 4; ++ks) S[0] = mma(Vb[ks], xl[4 * ks], S[0]);
            }
            static_for<0, NCQ>([&](auto ci) {
                constexpr int cc = decltype(ci)::value;
                constexpr int u0 = PT::u0(cc, GH);
                const float *xm = sm.xT + PT::chan(cc, GH, gw) * TS + h;
                float Bm[C / 4];
#pragma unroll
                for (int ks = 0; ks < C / 4; ++ks) Bm[ks] = xm[4 * ks] * Vb[ks];
                static_for<u0, NU>([&](auto ui) {
                    constexpr int u = decltype(ui)::value;
                    constexpr int t = PT::first(cc, GH) + u - u0;
#pragma unroll
                    for (int ks = 0; ks < C / 4; ++ks) S[t] = mma(Bm[ks], Ak[u][ks], S[t]);
                });
            });
            if (P == 1 && ylb >= 0 && tid < D) {
                float s = 0.f;
#pragma unroll 8
                for (int t = 0; t < C; ++t) s = fmaf(sm.wt[t], sm.xrow[t * RS + tid], s);
                y2reg += s;
            }
            if (P == 2 && ylb >= 0) {
                const float *xa = sm.xT + (16 * ylb + r16) * TS + h;
                float aw[C / 4];
#pragma unroll
                for (int ks = 0; ks < C / 4; ++ks) aw[ks] = xa[4 * ks] * sm.wt[4 * ks + h];
#pragma unroll
                for (int kk = 0; kk < NYW; ++kk) {
                    const int u2 = w + NW * kk;
                    if (u2 >= NU) break;
                    const float *xb = sm.xT + (16 * u2 + r16) * TS + h;
#pragma unroll
                    for (int ks = 0; ks < C / 4; ++ks) Y[kk] = mma(aw[ks], xb[4 * ks], Y[kk]);
                }
                if (tid < 16) {
                    float s = 0.f;
#pragma unroll 8
                    for (int t = 0; t < C; ++t) s = fmaf(sm.wt[t], sm.xrow[t * RS + 16 * ylb + tid], s);
                    y2reg += s;
                }
            }
            __syncthreads();
            if (P == 1 && ylb >= 0 && tid < D) sm.y2[tid] = y2reg;
            if (P == 2 && ylb >= 0) {
#pragma unroll
                for (int kk = 0; kk < NYW; ++kk) {
                    const int u2 = w + NW * kk;
                    if (u2 >= NU) break;
#pragma unroll
                    for (int i = 0; i < 4; ++i) sm.y3[(4 * h + i) * RS + 16 * u2 + r16] = Y[kk][i];
                }
                if (tid < 16) sm.y2[tid] = y2reg;
            }
        }
        __syncthreads();
    };
    with_wave_class<D, P>(gw, [&](auto ghc) {
        if constexpr (MODE == BOTH) {
            // non-causal, one segment: the totals first, then every output row
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
#pragma unroll
        for (int t = 0; t < NT; ++t) *(f4 *)(sum + ((size_t)(w * NT + t) * 64 + lane) * 4) = S[t];
        float *sy = sum + GS::STATE;
        for (int e = tid; e < GS::Y3N; e += NTH) sy[e] = sm.y3[(e / D) * RS + e % D];
        if (tid < GS::Y2N) sy[GS::Y3N + tid] = y2reg;
    }
}

// rg_i = 1 / G_i, c_i = (dO_i . O_i) / G_i; clears the float32 gradients.
// 16 threads per token.
template <int D, typename T>
__global__ __launch_bounds__(256) void bwd_prep_kernel(const T *__restrict__ o,
                                                       const T *__restrict__ dout,
                                                       const float *__restrict__ g,
                                                       float *__restrict__ rg,
                                                       float *__restrict__ cvec,
                                                       float *__restrict__ dqh,
                                                       float *__restrict__ dkh, size_t rows)
{
    const size_t r = (size_t)blockIdx.x * 16 + (threadIdx.x >> 4);
    const int j = threadIdx.x & 15;
    if (r >= rows) return;   // whole groups of 16 lanes
    float acc = 0.f;
#pragma unroll
    for (int i = 0; i < D / 16; ++i) {
        const size_t e = r * D + j + 16 * i;
        acc = fmaf(io<T>::ld(dout, e), io<T>::ld(o, e), acc);
        dqh[e] = 0.f;
        dkh[e] = 0.f;
    }
    acc += __shfl_xor(acc, 1);
    acc += __shfl_xor(acc, 2);
    acc += __shfl_xor(acc, 4);
    acc += __shfl_xor(acc, 8);
    if (j == 0) {
        const float G = g[r];
        rg[r] = 1.0f / G;
        cvec[r] = acc / G;
    }
}

// Back through Eqs. (6)-(7) and cast: dx = (dx^ - mean dx^ - x^ mean(dx^ x^)) / std,
// dx^ = sc dxh (the scans differentiate with respect to the scaled query
// tau q^).  blockIdx.y: 0 = dq, 1 = dk; 16 threads per token.
template <int D, typename T>
__global__ __launch_bounds__(256) void bwd_finish_kernel(const T *__restrict__ q,
                                                         const T *__restrict__ k,
                                                         const float *__restrict__ dqh,
                                                         const float *__restrict__ dkh,
                                                         T *__restrict__ dq, T *__restrict__ dk,
                                                         size_t rows, float qs)
{
    const int which = blockIdx.y;
    const T *x = which ? k : q;
    const float *dxh = which ? dkh : dqh;
    T *dx = which ? dk : dq;
    const float sc = which ? 1.0f : qs;
    const size_t r = (size_t)blockIdx.x * 16 + (threadIdx.x >> 4);
    const int j = threadIdx.x & 15;
    if (r >= rows) return;
    constexpr int CPT = D / 16;
    float xv[CPT], gv[CPT];
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
        const size_t e = r * D + j + 16 * i;
        xv[i] = io<T>::ld(x, e);
        gv[i] = sc * dxh[e];
        s += xv[i];
    }
    auto sum16 = [](float a) {
        a += __shfl_xor(a, 1);
        a += __shfl_xor(a, 2);
        a += __shfl_xor(a, 4);
        a += __shfl_xor(a, 8);
        return a;
    };
    const float mu = sum16(s) * (1.0f / D);
    float var = 0.f;
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
        xv[i] -= mu;
        var = fmaf(xv[i], xv[i], var);
    }
    const float rs = rsqrtf(sum16(var) * (1.0f / D));
    float m1 = 0.f, m2 = 0.f;
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
        xv[i] *= rs;
        m1 += gv[i];
        m2 = fmaf(gv[i], xv[i], m2);
    }
    m1 = sum16(m1) * (1.0f / D);
    m2 = sum16(m2) * (1.0f / D);
#pragma unroll
    for (int i = 0; i < CPT; ++i)
        io<T>::st(dx, r * D + j + 16 * i, (gv[i] - m1 - xv[i] * m2) * rs);
}

template <int D, int P>
struct BwdPlan {
    int items, nch, nseg;
    size_t vec_bytes, grad_bytes, scan_bytes;
    BwdPlan(int BH, int N)
    {
        items = BH * (D / SL) * Pat<D, P>::NPART;
        nch = (N + C - 1) / C;
        nseg = nseg_of(items, nch);
        const size_t rows = (size_t)BH * N;
        vec_bytes = a256(rows * 4);
        grad_bytes = a256(rows * D * 4);
        const size_t gsum = nseg > 1 ? a256((size_t)items * nseg * GSum<D, P>::BYTES) : 0;
        const size_t fwd = f32mfma_fwd_workspace(BH, N, D, P);   // the dv scan's
        scan_bytes = gsum > fwd ? gsum : fwd;
    }
    // rg, c, dq~, dk^, then the scans' region (used by one scan at a time)
    size_t bytes() const { return 2 * vec_bytes + 2 * grad_bytes + scan_bytes; }
};

template <int D, typename T, bool REV, int P>
hipError_t grad_launch(const BwdPlan<D, P> &pl, const T *X, const T *Z, const T *VS, const T *UC,
                       const float *vsm, const float *ucm, const float *wv, const float *zv,
                       float *outh, float *sums, int N, int causal, float xs, float zsc,
                       hipStream_t st)
{
    using GS = GSum<D, P>;
    const int items = pl.items, nseg = pl.nseg;
    if (!grid_fits((long long)items * nseg, Pat<D, P>::NTH)) return hipErrorInvalidConfiguration;
    const dim3 grid((unsigned)(items * nseg)), blk(Pat<D, P>::NTH);
    const size_t stride = GS::BYTES / 4;
    const dim3 pgrid((unsigned)((GS::FLOATS + 255) / 256), items);
    if (causal) {
        if (nseg > 1) {
            hipLaunchKernelGGL((grad_kernel<D, T, true, DELTA, REV, P>), grid, blk, 0, st, X, Z, VS,
                               UC, vsm, ucm, wv, zv, outh, sums, N, nseg, xs, zsc);
            hipLaunchKernelGGL(prefix_kernel, pgrid, dim3(256), 0, st, sums, nseg, GS::FLOATS,
                               stride, 1);
        }
        hipLaunchKernelGGL((grad_kernel<D, T, true, SCAN, REV, P>), grid, blk, 0, st, X, Z, VS, UC,
                           vsm, ucm, wv, zv, outh, sums, N, nseg, xs, zsc);
    } else if (nseg == 1) {
        hipLaunchKernelGGL((grad_kernel<D, T, false, BOTH, REV, P>), grid, blk, 0, st, X, Z, VS, UC,
                           vsm, ucm, wv, zv, outh, nullptr, N, nseg, xs, zsc);
    } else {
        hipLaunchKernelGGL((grad_kernel<D, T, false, DELTA, REV, P>), grid, blk, 0, st, X, Z, VS,
                           UC, vsm, ucm, wv, zv, outh, sums, N, nseg, xs, zsc);
        hipLaunchKernelGGL(prefix_kernel, pgrid, dim3(256), 0, st, sums, nseg, GS::FLOATS, stride,
                           0);
        hipLaunchKernelGGL((grad_kernel<D, T, false, QUERY, REV, P>), grid, blk, 0, st, X, Z, VS,
                           UC, vsm, ucm, wv, zv, outh, sums, N, nseg, xs, zsc);
    }
    return hipGetLastError();
}

template <int D, typename T, int P>
hipError_t bwd_run(const void *q, const void *k, const void *v, const void *o, const void *dout,
                   const float *g, void *dq, void *dk, void *dv, int BH, int N, int causal,
                   float qs, void *ws, hipStream_t st)
{
    const BwdPlan<D, P> pl(BH, N);
    const size_t rows = (size_t)BH * N;
    char *p = (char *)ws;
    float *rg = (float *)p;
    float *cvec = (float *)(p + pl.vec_bytes);
    float *dqh = (float *)(p + 2 * pl.vec_bytes);
    float *dkh = (float *)(p + 2 * pl.vec_bytes + pl.grad_bytes);
    void *scan = p + 2 * pl.vec_bytes + 2 * pl.grad_bytes;
    const size_t rb = (rows + 15) / 16;
    // every grid of the sequence checked before the first launch
    if (!grid_fits((long long)rb, 256) ||
        !grid_fits((long long)pl.items * pl.nseg, Pat<D, P>::NTH) ||
        !f32mfma_fwd_grids_fit(BH, N, D, P))
        return hipErrorInvalidConfiguration;
    const T *Q = (const T *)q, *K = (const T *)k, *V = (const T *)v, *DO = (const T *)dout;
    hipLaunchKernelGGL((bwd_prep_kernel<D, T>), dim3((unsigned)rb), dim3(256), 0, st, (const T *)o,
                       DO, g, rg, cvec, dqh, dkh, rows);
    hipError_t e = f32mfma_dv(q, k, dout, rg, dv, BH, N, D, P, causal,
                              std::is_same<T, bf16_t>::value, qs, scan, st);
    if (e != hipSuccess) return e;
    // dq~: X = k^, VS = v, w = 1; Z = tau q^, UC = dO / G, z = -c
    e = grad_launch<D, T, false, P>(pl, K, Q, V, DO, nullptr, rg, nullptr, cvec, dqh,
                                    (float *)scan, N, causal, 1.0f, qs, st);
    if (e != hipSuccess) return e;
    // dk^: X = tau q^, VS = dO / G, w = c; Z = k^, UC = v, z = -1 (reverse order)
    e = grad_launch<D, T, true, P>(pl, Q, K, DO, V, rg, nullptr, cvec, nullptr, dkh,
                                   (float *)scan, N, causal, qs, 1.0f, st);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((bwd_finish_kernel<D, T>), dim3((unsigned)rb, 2), dim3(256), 0, st, Q, K,
                       dqh, dkh, (T *)dq, (T *)dk, rows, qs);
    return hipGetLastError();
}

template <typename T, int P>
hipError_t bwd_dt(const void *q, const void *k, const void *v, const void *o, const void *dout,
                  const float *g, void *dq, void *dk, void *dv, int BH, int N, int D, int causal,
                  float qs, void *ws, hipStream_t st)
{
    switch (D) {
    case 16: return bwd_run<16, T, P>(q, k, v, o, dout, g, dq, dk, dv, BH, N, causal, qs, ws, st);
    case 32: return bwd_run<32, T, P>(q, k, v, o, dout, g, dq, dk, dv, BH, N, causal, qs, ws, st);
    case 64: return bwd_run<64, T, P>(q, k, v, o, dout, g, dq, dk, dv, BH, N, causal, qs, ws, st);
    case 128: return bwd_run<128, T, P>(q, k, v, o, dout, g, dq, dk, dv, BH, N, causal, qs, ws, st);
    }
    return hipErrorInvalidValue;
}

}  // namespace m32

size_t f32mfma_bwd_workspace(int BH, int N, int D, int p)
{
    using namespace m32;
    if (p == 1) {
        switch (D) {
        case 16: return BwdPlan<16, 1>(BH, N).bytes();
        case 32: return BwdPlan<32, 1>(BH, N).bytes();
        case 64: return BwdPlan<64, 1>(BH, N).bytes();
        case 128: return BwdPlan<128, 1>(BH, N).bytes();
        }
        return 0;
    }
    switch (D) {
    case 16: return BwdPlan<16, 2>(BH, N).bytes();
    case 32: return BwdPlan<32, 2>(BH, N).bytes();
    case 64: return BwdPlan<64, 2>(BH, N).bytes();
    case 128: return BwdPlan<128, 2>(BH, N).bytes();
    }
    return 0;
}

hipError_t f32mfma_bwd(const void *q, const void *k, const void *v, const void *o,
                       const void *dout, const float *g, void *dq, void *dk, void *dv, int BH,
                       int N, int D, int p, int causal, int is_bf16, float qs, void *ws,
                       hipStream_t st)
{
    using namespace m32;
    if (!f32mfma_applies(D, p, is_bf16)) return hipErrorInvalidValue;
    if (is_bf16)
        return p == 2 ? bwd_dt<bf16_t, 2>(q, k, v, o, dout, g, dq, dk, dv, BH, N, D, causal, qs, ws, st)
                      : bwd_dt<bf16_t, 1>(q, k, v, o, dout, g, dq, dk, dv, BH, N, D, causal, qs, ws, st);
    return p == 2 ? bwd_dt<float, 2>(q, k, v, o, dout, g, dq, dk, dv, BH, N, D, causal, qs, ws, st)
                  : bwd_dt<float, 1>(q, k, v, o, dout, g, dq, dk, dv, BH, N, D, causal, qs, ws, st);
}

}  // namespace fm

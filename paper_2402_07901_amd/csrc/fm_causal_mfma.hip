// Causal Fastmax forward on CDNA4 MFMA, head dimension 64, p = 2, bf16 I/O.
//
// Chunked causal scan (Sec. 2.4, causal moments "xcausal"/"ycausal" carried
// across chunks of 128 tokens instead of per row).  One workgroup owns one
// (batch, head, slice of 16 value columns); its eight waves hold the moment
// state S[f][j] = sum_n phi_f(k^_n) v_nj of the slice as fp32 MFMA
// accumulators for the whole sequence, so the state never touches HBM.
//
// Features: the 21-tile-per-wave pattern of fm_mfma.h (symmetric 16x16
// tiles of k_m k_l plus the linear tiles); 84 accumulator registers per lane.
//
// Per chunk:
//  (i)  query contraction F^T += S^T Psi(Q)^T.  The accumulator layout of a
//       16x16 MFMA tile (lane: column j, rows 4h..4h+3) is used directly as
//       the A operand of the next MFMA by pairing two tiles per 32-wide K
//       step (K index 8h+r <-> tile a row 4h+r, 8h+4+r <-> tile b row 4h+r);
//       the Psi operand is generated in registers with packed fp16 multiplies
//       in the same K order.  Each wave contracts its own tiles for all 128
//       tokens; partial F^T go through LDS.
//  (ii) in-chunk block tril(f(Q K^T)) V on MFMA, and the denominator
//       G_i = n0 + q.y2 + 1/2 q^T Y3 q + in-chunk row sums, with Y3 = sum k k^T
//       kept as 10 symmetric fp32 accumulator tiles.
//  (iii) state update S += Phi(K)^T V per m: A = K^T tiles, B = diag(k_m) V
//       generated with packed multiplies.
//
// Operands are fp16 (q^, k^ are standardised so |x| <= 8).  v is scaled by a
// power of two 2^-e chosen per workgroup from max|v| so that every state
// entry (bounded by N * 63 * max|v|) stays below 2^15; the output is scaled
// back.  Y3 is converted with its own power of two per chunk.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "fm_common.h"
#include "fm_internal.h"
#include "fm_mfma.h"

namespace fm {
namespace mfma_causal {

using namespace mx;

constexpr int C = 128;        // tokens per chunk
constexpr int NRT = C / 16;   // 16-token row tiles per chunk
constexpr int NKS2 = C / 32;  // 32-token K steps of the state update
constexpr int NW = 8;         // waves per workgroup (2 per SIMD)
constexpr int NTH = NW * 64;
constexpr int SL = 16;        // value columns per workgroup
constexpr int NSL = D / SL;

struct Smem {
    _Float16 qrow[C * RS64];        // q^ [token][m]
    _Float16 krow[C * RS64];        // k^ [token][m]
    _Float16 kT[2][D * RS128];      // k^ [m][token], double-buffered by chunk parity
    _Float16 vT[2][SL * RS128];     // scaled v [j][token], double-buffered
    _Float16 y3h[D * RS64];         // scaled Y3 (prefix before the chunk)
    float fpart[NW * C * SL];       // partial F^T: [wave][column quad][token][4]
    float gpart[NW * C];            // partial denominators: [wave][token]
    float y2[2][D];                 // sum k^ before the chunk (by chunk parity)
    float y2c[D];                   // this chunk's sum k^
    float x1[2][SL];                // sum of scaled v before the chunk
    float x1c[SL];
    float red[NW];
};

// DV = false: the forward O = F / G.  DV = true: the reverse-causal
// numerator of the backward, dv_n = sum_{i >= n} f(k^_n . q^_i) u_i with
// u_i = dO_i / G_i (Sec. 2.5): the scan runs over the tokens in reverse order
// (logical token n is row N-1-n), q and k trade roles (the caller passes k as
// q and q as k), v is dO scaled per row by rg = 1/G, and F is stored without
// the divide; the denominator terms are skipped.
template <bool DV>
__device__ __forceinline__ void run_scan(Smem &sm, const bf16_t *__restrict__ q,
                                         const bf16_t *__restrict__ k,
                                         const bf16_t *__restrict__ v, bf16_t *__restrict__ out,
                                         float *__restrict__ g, const float *__restrict__ rg,
                                         int N, int sl, int vexp)
{
    const int w = threadIdx.x >> 6;    // wave
    const bool has_lin = w < 4;

    f4 acc[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = f4{0.f, 0.f, 0.f, 0.f};
    f4 y3acc[2] = {f4{0.f, 0.f, 0.f, 0.f}, f4{0.f, 0.f, 0.f, 0.f}};
    int y3u[2], y3u2[2];
    y3_tile(w, 0, y3u[0], y3u2[0]);
    y3_tile(w, w < 2 ? 1 : 0, y3u[1], y3u2[1]);
    const int ny3 = y3_count(w);

    const float vscale = ldexpf(1.0f, -vexp);   // v -> v * 2^-e
    const float oscale = ldexpf(1.0f, vexp);
    int gexp = 0;                                // Y3 in LDS is Y3 * 2^-gexp
    const int nch = (N + C - 1) / C;

    // Lane-derived LDS offsets are recomputed in every phase from an opaque
    // copy of the thread id: hoisted out of the loop they would stay live for
    // the whole scan and spill.
    int tid = threadIdx.x;
    int lane = tid & 63, r16 = lane & 15, h = lane >> 4;
    // loader roles: tokens 2*tg, 2*tg+1, channels 8*cg .. 8*cg+7
    int tg = tid >> 3, cg = tid & 7;
    int vt = tid >> 1, vh = tid & 1;             // v (tid < 256): token vt, columns 8*vh..
    auto refresh_ids = [&]() {
        asm volatile("" : "+v"(tid));
        lane = tid & 63;
        r16 = lane & 15;
        h = lane >> 4;
        tg = tid >> 3;
        cg = tid & 7;
        vt = tid >> 1;
        vh = tid & 1;
    };

    uint4 pq[2], pk[2], pv;
    float prg = 1.0f;   // DV: 1/G of the v row
    auto prefetch = [&](int c) {
        const uint4 z = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int n = c * C + 2 * tg + j;
            pq[j] = pk[j] = z;
            if (n < N) {
                const size_t pn = DV ? (size_t)(N - 1 - n) : (size_t)n;
                pq[j] = *(const uint4 *)(q + pn * D + 8 * cg);
                pk[j] = *(const uint4 *)(k + pn * D + 8 * cg);
            }
        }
        const int nv = c * C + vt;
        pv = z;
        if (tid < 2 * C && nv < N) {
            const size_t pn = DV ? (size_t)(N - 1 - nv) : (size_t)nv;
            pv = *(const uint4 *)(v + pn * D + SL * sl + 8 * vh);
            if constexpr (DV) prg = rg[pn];
        }
    };
    // Staging of chunk c (Sec. 2.2, Eqs. 6-7): standardise q and k rows, store
    // q^, k^ (row-major), k^ transposed and the scaled v transposed.
    auto stage_q = [&](int c) {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int row = 2 * tg + j;
            float x[8];
            bf16x8_to_f32(pq[j], x);
            *(h8 *)(sm.qrow + sw64(row, 8 * cg)) = standardise8(x, c * C + row < N);
        }
    };
    auto stage_kv = [&](int c) {
        const int buf = c & 1;
        h8 hk[2];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int row = 2 * tg + j;
            float x[8];
            bf16x8_to_f32(pk[j], x);
            hk[j] = standardise8(x, c * C + row < N);
            *(h8 *)(sm.krow + sw64(row, 8 * cg)) = hk[j];
        }
#pragma unroll
        for (int i = 0; i < 8; ++i)
            *(h2 *)(sm.kT[buf] + sw128(8 * cg + i, 2 * tg)) = h2{hk[0][i], hk[1][i]};
        if (tid < 2 * C) {
            float xv[8];
            bf16x8_to_f32(pv, xv);
            const float vs = DV ? vscale * prg : vscale;
#pragma unroll
            for (int i = 0; i < 8; ++i)
                sm.vT[buf][sw128(8 * vh + i, vt)] = (_Float16)(xv[i] * vs);
        }
    };

    // prologue: stage chunk 0
    prefetch(0);
    stage_q(0);
    stage_kv(0);
    __syncthreads();

    for (int c = 0; c < nch; ++c) {
        const int n0 = c * C;
        const int nvalid = min(C, N - n0);
        const int cur = c & 1, nxt = cur ^ 1;

        // ---- (I) query contraction, in-chunk block and denominators ---------
        __builtin_amdgcn_sched_barrier(0);
        refresh_ids();
        {
            // state -> fp16 A operands, two tiles per K step; diagonal tiles
            // carry the 1/2 of f_2's quadratic term
            h8 Ast[NKS];
            static_for<0, NKS>([&](auto pi) {
                constexpr int p = decltype(pi)::value;
                constexpr int ta = 2 * p, tb = 2 * p + 1;
                h4 a = cvt4(acc[ta]);
                if constexpr (is_diag(ta)) a = scale4(a, (_Float16)0.5f);
                h4 b = h4{0, 0, 0, 0};
                if constexpr (tb < NT) {
                    b = cvt4(acc[tb < NT ? tb : 0]);
                    if constexpr (is_diag(tb)) b = scale4(b, (_Float16)0.5f);
                }
                Ast[p] = cat(a, b);
            });

            const _Float16 *kTc = sm.kT[cur];
            const _Float16 *vTc = sm.vT[cur];
#pragma unroll 1
            for (int rt = 0; rt < NRT; ++rt) {
                const int tok = 16 * rt + r16;
                h4 myl[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) myl[u] = ld4(sm.qrow + sw64(tok, 16 * u + 4 * h));
                // linear features l = 16w + 4h + r (zero state in waves 4..7)
                const h4 mylin = ld4(sm.qrow + sw64(tok, 16 * (w & 3) + 4 * h));
                // the wave's channels m = w + 8*idx
                _Float16 qm[8];
#pragma unroll
                for (int idx = 0; idx < 8; ++idx) qm[idx] = sm.qrow[sw64(tok, w + 8 * idx)];
                f4 F0 = {0.f, 0.f, 0.f, 0.f}, F1 = {0.f, 0.f, 0.f, 0.f};
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
                    if constexpr (p & 1) F1 = mfma(Ast[p], B, F1);
                    else F0 = mfma(Ast[p], B, F0);
                });
                // In-chunk tril block.  Row tile rt has rt/2 + 1 items (pairs of
                // 16-token key tiles); the chunk's 20 items are dealt round-robin
                // to the 8 waves.  Each item: two S^T tiles (rows t, cols i = tok),
                // their weights f(s) and one MFMA F^T += V^T W^T.
                const int ibase = (rt / 2) * (rt / 2 + 1) + ((rt & 1) ? rt / 2 + 1 : 0);
                const int first = (w - ibase % NW + NW) % NW;   // first item j of this wave
                float gpart = 0.f;
                if (first <= rt / 2 || (!DV && rt == w)) {
                    const h8 QB0 = ld8(sm.qrow + sw64(tok, 8 * h));
                    const h8 QB1 = ld8(sm.qrow + sw64(tok, 32 + 8 * h));
                    auto wtile = [&](int tt) -> h4 {
                        f4 S = {0.f, 0.f, 0.f, 0.f};
                        S = mfma(ld8(sm.krow + sw64(16 * tt + r16, 8 * h)), QB0, S);
                        S = mfma(ld8(sm.krow + sw64(16 * tt + r16, 32 + 8 * h)), QB1, S);
                        f4 wv;
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            const float x = S[i];
                            float y = fmaf(0.5f * x, x, 1.0f + x);
                            if (tt == rt && (4 * h + i) > r16) y = 0.0f;
                            wv[i] = y;
                            gpart += y;
                        }
                        return cvt4(wv);
                    };
                    for (int j = first; j <= rt / 2; j += NW) {
                        const int a = 2 * j, b = a + 1;
                        const h4 wa = wtile(a);
                        const h4 va = ld4(vTc + sw128(r16, 16 * a + 4 * h));
                        h4 wb = h4{0, 0, 0, 0}, vb = h4{0, 0, 0, 0};
                        if (b <= rt) {
                            wb = wtile(b);
                            vb = ld4(vTc + sw128(r16, 16 * b + 4 * h));
                        }
                        F0 = mfma(cat(va, vb), cat(wa, wb), F0);
                    }
                    if (!DV && rt == w) {
                        // inter-chunk denominator q.y2 + 1/2 q^T Y3 q (+ n0)
                        float gq = 0.f;
                        const float ys = ldexpf(2.0f, -gexp);
#pragma unroll
                        for (int cc = 0; cc < 4; ++cc) {
                            f4 T;
#pragma unroll
                            for (int i = 0; i < 4; ++i) T[i] = ys * sm.y2[cur][16 * cc + 4 * h + i];
                            T = mfma(ld8(sm.y3h + sw64(16 * cc + r16, 8 * h)), QB0, T);
                            T = mfma(ld8(sm.y3h + sw64(16 * cc + r16, 32 + 8 * h)), QB1, T);
#pragma unroll
                            for (int i = 0; i < 4; ++i) gq = fmaf((float)myl[cc][i], T[i], gq);
                        }
                        gpart = fmaf(0.5f * ldexpf(1.0f, gexp), gq, gpart);
                        if (h == 0) gpart += (float)n0;
                    }
                    gpart += __shfl_xor(gpart, 16);
                    gpart += __shfl_xor(gpart, 32);
                }
                if (h == 0) sm.gpart[w * C + tok] = gpart;
                *(f4 *)(sm.fpart + ((w * 4 + h) * C + tok) * 4) = F0 + F1;
            }
            // this chunk's sums of k^ (for y2, waves 0-3) and of scaled v (x1, wave 4)
            if (!DV && w < 4) {
                const int m = 16 * w + r16;
                float s = 0.f;
#pragma unroll
                for (int cc = 0; cc < 4; ++cc) s += hsum8(ld8(kTc + sw128(m, 32 * h + 8 * cc)));
                s += __shfl_xor(s, 16);
                s += __shfl_xor(s, 32);
                if (h == 0) sm.y2c[m] = s;
            } else if (w == 4) {
                float sv = 0.f;
#pragma unroll
                for (int cc = 0; cc < 4; ++cc) sv += hsum8(ld8(vTc + sw128(r16, 32 * h + 8 * cc)));
                sv += __shfl_xor(sv, 16);
                sv += __shfl_xor(sv, 32);
                if (h == 0) sm.x1c[r16] = sv;
            }
        }
        __syncthreads();

        // ---- (M) output of chunk c, state update with chunk c, staging of c+1 --
        __builtin_amdgcn_sched_barrier(0);
        refresh_ids();
        {
            // combine partials, divide, store
            const int tok = tid & (C - 1), cq = tid >> 7;
            f4 F = *(const f4 *)(sm.x1[cur] + 4 * cq);
            float Gi = 0.f;
#pragma unroll
            for (int ww = 0; ww < NW; ++ww) {
                F += *(const f4 *)(sm.fpart + ((ww * 4 + cq) * C + tok) * 4);
                Gi += sm.gpart[ww * C + tok];
            }
            if (n0 + tok < N) {
                const float sc = DV ? oscale : oscale * __builtin_amdgcn_rcpf(Gi);
                uint2 o;
                o.x = pack_bf16x2(F[0] * sc, F[1] * sc);
                o.y = pack_bf16x2(F[2] * sc, F[3] * sc);
                const size_t pn = DV ? (size_t)(N - 1 - (n0 + tok)) : (size_t)(n0 + tok);
                *(uint2 *)(out + pn * D + SL * sl + 4 * cq) = o;
                if (!DV && g && sl == 0 && cq == 0) g[n0 + tok] = Gi;
            }
            // prefixes for the next chunk
            if (tid < D) sm.y2[nxt][tid] = sm.y2[cur][tid] + sm.y2c[tid];
            else if (tid < D + SL) sm.x1[nxt][tid - D] = sm.x1[cur][tid - D] + sm.x1c[tid - D];
        }
        const bool more = c + 1 < nch;
        if (more) prefetch(c + 1);
        {
            // state update S += Phi(K)^T V, Y3 += K^T K, interleaved with the
            // staging of the next chunk (its loads land behind the first steps)
            const _Float16 *kTc = sm.kT[cur];
            const _Float16 *vTc = sm.vT[cur];
            auto ustep = [&](int s) {
                h8 Ak[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) Ak[u] = ld8(kTc + sw128(16 * u + r16, 32 * s + 8 * h));
                const h8 Vf = ld8(vTc + sw128(r16, 32 * s + 8 * h));
                if (has_lin)   // linear tile: x2[l][j] += sum_t k_tl v_tj, l in tile w
                    acc[0] = mfma(ld8(kTc + sw128(16 * w + r16, 32 * s + 8 * h)), Vf, acc[0]);
                static_for<0, 8>([&](auto ii) {
                    constexpr int idx = decltype(ii)::value;
                    constexpr int u0 = u0_of(idx);
                    constexpr int t0 = first_tile(idx);
                    const int m = w + 8 * idx;
                    const h8 km = ld8(kTc + sw128(m, 32 * s + 8 * h));
                    const h8 Wm = km * Vf;
                    static_for<u0, 4>([&](auto ui) {
                        constexpr int u = decltype(ui)::value;
                        acc[t0 + (u - u0)] = mfma(Ak[u], Wm, acc[t0 + (u - u0)]);
                    });
                });
#pragma unroll
                for (int kk = 0; kk < 2; ++kk)
                    if (!DV && kk < ny3)
                        y3acc[kk] = mfma(ld8(kTc + sw128(16 * y3u[kk] + r16, 32 * s + 8 * h)),
                                         ld8(kTc + sw128(16 * y3u2[kk] + r16, 32 * s + 8 * h)),
                                         y3acc[kk]);
            };
            ustep(0);
            ustep(1);
            ustep(2);
            if (more) stage_q(c + 1);
            ustep(3);
            if (more) stage_kv(c + 1);
            // scaled fp16 copy of Y3 for the next chunk's denominators
            const int gnext = max(0, pow2_exponent(64.0f * (float)(n0 + nvalid)));
            const float gs = ldexpf(1.0f, -gnext);
#pragma unroll
            for (int kk = 0; kk < 2; ++kk) {
                if (DV || kk >= ny3) break;
                const int u = y3u[kk], u2 = y3u2[kk];
                // lane: column m = 16*u2 + r16, rows l = 16*u + 4h + i
                const int mcol = 16 * u2 + r16;
                h4 hv;
#pragma unroll
                for (int i = 0; i < 4; ++i) hv[i] = (_Float16)(y3acc[kk][i] * gs);
                *(h4 *)(sm.y3h + sw64(mcol, 16 * u + 4 * h)) = hv;       // Y3[m][l]
                if (u != u2) {
#pragma unroll
                    for (int i = 0; i < 4; ++i) sm.y3h[sw64(16 * u + 4 * h + i, mcol)] = hv[i];
                }
            }
            gexp = gnext;
        }
        __syncthreads();
    }
}

template <bool DV>
__global__ __launch_bounds__(NTH, 2) void fwd_causal_kernel(const bf16_t *__restrict__ q,
                                                            const bf16_t *__restrict__ k,
                                                            const bf16_t *__restrict__ v,
                                                            bf16_t *__restrict__ out,
                                                            float *__restrict__ g,
                                                            const float *__restrict__ rg, int N,
                                                            int BH)
{
    extern __shared__ __align__(16) unsigned char smem_raw[];
    Smem &sm = *reinterpret_cast<Smem *>(smem_raw);

    // XCD-aware mapping: consecutive block ids land on different XCDs
    // (round-robin over 8); keep the 4 slices of a head on one XCD so that
    // its q and k rows are shared through that XCD's L2.
    const int nblk = gridDim.x;
    const int b = blockIdx.x;
    int head, sl;
    if ((nblk & 31) == 0) {
        const int xcd = b & 7, idx = b >> 3;
        sl = idx & 3;
        head = (idx >> 2) * 8 + xcd;
    } else {
        head = b / NSL;
        sl = b % NSL;
    }
    if (head >= BH) return;
    const size_t hb = (size_t)head * N * D;
    q += hb;
    k += hb;
    v += hb;
    out += hb;
    if (g) g += (size_t)head * N;
    if (rg) rg += (size_t)head * N;

    // max |v| over this slice -> power-of-two scale
    const int tid = threadIdx.x;
    float vmax = 0.f;
    for (int p = tid; p < 2 * N; p += NTH) {
        const int n = p >> 1, hh = p & 1;
        float x[8];
        bf16x8_to_f32(*(const uint4 *)(v + (size_t)n * D + SL * sl + 8 * hh), x);
        const float r = DV ? fabsf(rg[n]) : 1.0f;
#pragma unroll
        for (int i = 0; i < 8; ++i) vmax = fmaxf(vmax, fabsf(x[i]) * r);
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) vmax = fmaxf(vmax, __shfl_xor(vmax, o));
    if ((tid & 63) == 0) sm.red[tid >> 6] = vmax;
    if (tid < D) { sm.y2[0][tid] = 0.f; sm.y2c[tid] = 0.f; }
    if (tid < SL) { sm.x1[0][tid] = 0.f; sm.x1c[tid] = 0.f; }
    for (int e = tid; e < D * RS64; e += NTH) sm.y3h[e] = (_Float16)0.0f;
    __syncthreads();
    vmax = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) vmax = fmaxf(vmax, sm.red[w]);
    const int vexp = pow2_exponent(vmax * 63.0f * (float)N);

    run_scan<DV>(sm, q, k, v, out, g, rg, N, sl, vexp);
}

}  // namespace mfma_causal

size_t mfma_causal_smem_bytes() { return sizeof(mfma_causal::Smem); }

hipError_t mfma_causal_fwd(const void *q, const void *k, const void *v, void *out, float *g,
                           int BH, int N, hipStream_t st)
{
    using namespace mfma_causal;
    static_assert(sizeof(Smem) <= 160 * 1024, "LDS budget");
    const size_t smem = sizeof(Smem);
    hipError_t e = hipFuncSetAttribute((const void *)fwd_causal_kernel<false>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(fwd_causal_kernel<false>, dim3(BH * NSL), dim3(NTH), smem, st,
                       (const bf16_t *)q, (const bf16_t *)k, (const bf16_t *)v, (bf16_t *)out, g,
                       (const float *)nullptr, N, BH);
    return hipGetLastError();
}

hipError_t mfma_causal_dv(const void *q, const void *k, const void *dout, const float *rg,
                          void *dv, int BH, int N, hipStream_t st)
{
    using namespace mfma_causal;
    const size_t smem = sizeof(Smem);
    hipError_t e = hipFuncSetAttribute((const void *)fwd_causal_kernel<true>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    if (e != hipSuccess) return e;
    // queries of this scan are the keys k (and vice versa), values dO / G
    hipLaunchKernelGGL(fwd_causal_kernel<true>, dim3(BH * NSL), dim3(NTH), smem, st,
                       (const bf16_t *)k, (const bf16_t *)q, (const bf16_t *)dout, (bf16_t *)dv,
                       (float *)nullptr, rg, N, BH);
    return hipGetLastError();
}

}  // namespace fm

// Causal Fastmax forward on CDNA4 MFMA, head dimension 64, p = 2, bf16 I/O.
//
// Chunked causal scan (Sec. 2.4, causal moments "xcausal"/"ycausal" carried
// across chunks of C tokens instead of per row).  One workgroup owns one
// (batch, head, slice of 16 value columns); its four waves hold the moment
// state S[f][j] = sum_n phi_f(k^_n) v_nj of the slice as fp32 MFMA
// accumulators for the whole sequence, so the state never touches HBM.
//
// Features.  The quadratic features k_m k_l are grouped in 16x16 tiles
// (m, u): rows l = 16u..16u+15 for one m, with u >= m/16 (symmetric tiles:
// 160 of them) plus 4 linear tiles (k_l) -- 2624 feature rows instead of the
// 4160 of the full square, 2080 + 65 being the minimum.  A "diagonal" tile
// (u == m/16) carries both (m,l) and (l,m) and is accumulated with weight 1/2;
// the others with weight 1, so psi(q).phi(k) = 1 + s + s^2/2 exactly
// (constant term separate).  Wave w owns the tiles of m = w (mod 4) and the
// linear tile u = w: 41 tiles, 164 accumulator registers.
//
// Per chunk:
//  (i)  query contraction F^T += S^T Psi(Q)^T.  The accumulator layout of a
//       16x16 MFMA tile (lane: column j, rows 4h..4h+3) is used directly as
//       the A operand of the next MFMA by pairing two tiles per 32-wide K
//       step (K index 8h+r <-> tile a row 4h+r, 8h+4+r <-> tile b row 4h+r);
//       the Psi operand is generated in registers with packed fp16 multiplies
//       in the same K order.  Each wave contracts its own tiles for all 64
//       tokens; partial F^T go through LDS.
//  (ii) in-chunk block tril(f(Q K^T)) V on MFMA, and the denominator
//       G_i = n0 + q.y2 + 1/2 q^T Y3 q + in-chunk row sums, with Y3 = sum k k^T
//       kept as 10 symmetric fp32 accumulator tiles.
//  (iii) state update S += Phi(K)^T V per m: A = K^T tiles (1/2 K^T for the
//       diagonal tile), B = diag(k_m) V generated with packed multiplies.
//
// Operands are fp16 (q^, k^ are standardised so |x| <= 8).  v is scaled by a
// power of two 2^-e chosen per workgroup from max|v| so that every state
// entry (bounded by N * 63 * max|v|) stays below 2^15; the output is scaled
// back.  Y3 is converted with its own power of two per chunk.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "fm_common.h"
#include "fm_internal.h"

namespace fm {
namespace mfma_causal {

typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef _Float16 h4 __attribute__((ext_vector_type(4)));
typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int D = 64;
constexpr int C = 64;         // tokens per chunk
constexpr int NW = 4;         // waves per workgroup
constexpr int NTH = NW * 64;
constexpr int SL = 16;        // value columns per workgroup
constexpr int NSL = D / SL;
constexpr int NT = 41;        // state tiles per wave
constexpr int NKS = (NT + 1) / 2;  // K steps of the query contraction
constexpr int RS = D + 8;     // padded LDS row stride (halves)

template <int I, int N, typename F>
__device__ __forceinline__ void static_for(F &&f)
{
    if constexpr (I < N) {
        f(std::integral_constant<int, I>{});
        static_for<I + 1, N>(f);
    }
}

struct Tile {
    int kind;  // 0 linear, 1 quadratic, -1 padding
    int m;     // channel m (quadratic) or -1
    int idx;   // position of m in the wave's m list
    int u;     // l tile
};

// t-th tile of wave W: t = 0 is the linear tile u = W; then for the wave's
// channels m = W, W+4, ..., W+60 the tiles u = m/16 .. 3.
__host__ __device__ constexpr Tile tile_of(int W, int t)
{
    if (t == 0) return Tile{0, -1, -1, W};
    int r = t - 1;
    for (int idx = 0; idx < 16; ++idx) {
        int m = W + 4 * idx;
        int n = 4 - m / 16;
        if (r < n) return Tile{1, m, idx, m / 16 + r};
        r -= n;
    }
    return Tile{-1, -1, -1, -1};
}

// first tile index of channel list position idx for wave W
__host__ __device__ constexpr int first_tile(int W, int idx)
{
    int t = 1;
    for (int i = 0; i < idx; ++i) t += 4 - (W + 4 * i) / 16;
    return t;
}

// Y3 tiles (u <= u2) owned by wave W
__host__ __device__ constexpr int y3_count(int W) { return W < 2 ? 3 : 2; }
__host__ __device__ constexpr int y3_u(int W, int k)
{
    constexpr int us[10] = {0, 0, 0, 0, 1, 1, 1, 2, 2, 3};
    return us[(W < 2 ? 3 * W : 6 + 2 * (W - 2)) + k];
}
__host__ __device__ constexpr int y3_u2(int W, int k)
{
    constexpr int us[10] = {0, 1, 2, 3, 1, 2, 3, 2, 3, 3};
    return us[(W < 2 ? 3 * W : 6 + 2 * (W - 2)) + k];
}

struct Smem {
    _Float16 qrow[C * RS];    // q^ row-major
    _Float16 qperm[C * RS];   // q^ with channel m at (m % 4) * 16 + m / 4
    _Float16 krow[C * RS];    // k^ row-major
    _Float16 kT[D * RS];      // k^ transposed [m][token]
    _Float16 vT[SL * RS];     // scaled v transposed [j][token]
    _Float16 y3h[D * RS];     // scaled Y3 (prefix before the chunk)
    float fpart[NW * C * SL]; // partial F^T per wave: [wave][token][j]
    float y2[D];              // sum k^ before the chunk
    float y2c[D];             // this chunk's sum k^
    float x1[SL];             // sum of scaled v before the chunk
    float x1c[SL];
    float g[C];
    float red[NW];
};

__device__ __forceinline__ f4 mfma(h8 a, h8 b, f4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ h4 cvt4(f4 x)
{
    h2 lo = {(_Float16)x[0], (_Float16)x[1]};
    h2 hi = {(_Float16)x[2], (_Float16)x[3]};
    return h4{lo[0], lo[1], hi[0], hi[1]};
}

__device__ __forceinline__ h8 cat(h4 a, h4 b)
{
    return h8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
}

__device__ __forceinline__ h4 scale4(h4 x, _Float16 s)
{
    h2 ss = {s, s};
    h2 lo = h2{x[0], x[1]} * ss;
    h2 hi = h2{x[2], x[3]} * ss;
    return h4{lo[0], lo[1], hi[0], hi[1]};
}

__device__ __forceinline__ h8 ld8(const _Float16 *p) { return *(const h8 *)p; }
__device__ __forceinline__ h4 ld4(const _Float16 *p) { return *(const h4 *)p; }

// 8 bf16 (one 16-byte load) -> 8 floats
__device__ __forceinline__ void bf16x8_to_f32(uint4 u, float *x)
{
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        x[2 * i] = __uint_as_float(w[i] << 16);
        x[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
}

// Smallest e with bound * 2^-e <= 2^15 (e may be negative), clamped.
__device__ __forceinline__ int pow2_exponent(float bound)
{
    if (!(bound > 0.0f)) return 0;
    int e = (int)ceilf(log2f(bound)) - 15;
    return e < -100 ? -100 : (e > 100 ? 100 : e);
}

template <int W>
__device__ __forceinline__ void run_wave(Smem &sm, const bf16_t *__restrict__ q,
                                         const bf16_t *__restrict__ k,
                                         const bf16_t *__restrict__ v, bf16_t *__restrict__ out,
                                         float *__restrict__ g, int N, int sl, int vexp)
{
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int r16 = lane & 15;
    const int h = lane >> 4;

    f4 acc[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = f4{0.f, 0.f, 0.f, 0.f};
    constexpr int NY = y3_count(W);
    f4 y3acc[NY];
#pragma unroll
    for (int t = 0; t < NY; ++t) y3acc[t] = f4{0.f, 0.f, 0.f, 0.f};

    const float vscale = ldexpf(1.0f, -vexp);   // v -> v * 2^-e
    const float oscale = ldexpf(1.0f, vexp);
    int gexp = 0;                                // Y3 in LDS is Y3 * 2^-gexp
    const int nch = (N + C - 1) / C;

    // loader roles: row r, quarter qq (16 channels) of q and k
    const int lr = tid >> 2, lq = tid & 3;
    const int vr = tid >> 1, vh = tid & 1;       // v loader (tid < 128)

    uint4 pq0, pq1, pk0, pk1, pv;
    auto prefetch = [&](int c) {
        const int n = c * C + lr;
        const uint4 z = {0u, 0u, 0u, 0u};
        pq0 = pq1 = pk0 = pk1 = pv = z;
        if (n < N) {
            const uint4 *qp = (const uint4 *)(q + (size_t)n * D + 16 * lq);
            const uint4 *kp = (const uint4 *)(k + (size_t)n * D + 16 * lq);
            pq0 = qp[0];
            pq1 = qp[1];
            pk0 = kp[0];
            pk1 = kp[1];
        }
        const int nv = c * C + vr;
        if (tid < 128 && nv < N)
            pv = *(const uint4 *)(v + (size_t)nv * D + SL * sl + 8 * vh);
    };
    prefetch(0);

    for (int c = 0; c < nch; ++c) {
        const int n0 = c * C;
        const int nvalid = min(C, N - n0);
        // ---- fold the previous chunk's sums into the prefixes ----------------
        if (c > 0) {
            if (tid < D) sm.y2[tid] += sm.y2c[tid];
            else if (tid < D + SL) sm.x1[tid - D] += sm.x1c[tid - D];
        }
        // ---- (L) standardise q, k (Sec. 2.2, Eqs. 6-7) and stage the chunk ----
        {
            const bool valid = (n0 + lr) < N;
            float xq[16], xk[16];
            bf16x8_to_f32(pq0, xq);
            bf16x8_to_f32(pq1, xq + 8);
            bf16x8_to_f32(pk0, xk);
            bf16x8_to_f32(pk1, xk + 8);
            float sq = 0.f, sk = 0.f;
#pragma unroll
            for (int i = 0; i < 16; ++i) { sq += xq[i]; sk += xk[i]; }
            sq += __shfl_xor(sq, 1);
            sq += __shfl_xor(sq, 2);
            sk += __shfl_xor(sk, 1);
            sk += __shfl_xor(sk, 2);
            const float mq = sq * (1.0f / D), mk = sk * (1.0f / D);
            float vq = 0.f, vk = 0.f;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                xq[i] -= mq;
                xk[i] -= mk;
                vq = fmaf(xq[i], xq[i], vq);
                vk = fmaf(xk[i], xk[i], vk);
            }
            vq += __shfl_xor(vq, 1);
            vq += __shfl_xor(vq, 2);
            vk += __shfl_xor(vk, 1);
            vk += __shfl_xor(vk, 2);
            const float rq = valid ? rsqrtf(vq * (1.0f / D)) : 0.0f;
            const float rk = valid ? rsqrtf(vk * (1.0f / D)) : 0.0f;
            _Float16 hq[16], hk[16];
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                hq[i] = (_Float16)(xq[i] * rq);
                hk[i] = (_Float16)(xk[i] * rk);
            }
            _Float16 *qr = sm.qrow + lr * RS + 16 * lq;
            _Float16 *kr = sm.krow + lr * RS + 16 * lq;
            *(h8 *)qr = h8{hq[0], hq[1], hq[2], hq[3], hq[4], hq[5], hq[6], hq[7]};
            *(h8 *)(qr + 8) = h8{hq[8], hq[9], hq[10], hq[11], hq[12], hq[13], hq[14], hq[15]};
            *(h8 *)kr = h8{hk[0], hk[1], hk[2], hk[3], hk[4], hk[5], hk[6], hk[7]};
            *(h8 *)(kr + 8) = h8{hk[8], hk[9], hk[10], hk[11], hk[12], hk[13], hk[14], hk[15]};
#pragma unroll
            for (int a = 0; a < 4; ++a)
                *(h4 *)(sm.qperm + lr * RS + a * 16 + 4 * lq) =
                    h4{hq[a], hq[a + 4], hq[a + 8], hq[a + 12]};
#pragma unroll
            for (int i = 0; i < 16; ++i) sm.kT[(16 * lq + i) * RS + lr] = hk[i];
            if (tid < 128) {
                float xv[8];
                bf16x8_to_f32(pv, xv);
#pragma unroll
                for (int i = 0; i < 8; ++i)
                    sm.vT[(8 * vh + i) * RS + vr] = (_Float16)(xv[i] * vscale);
            }
        }
        __syncthreads();
        if (c + 1 < nch) prefetch(c + 1);

        // ---- (I) query contraction, in-chunk block and denominators ---------
        {
            // state -> fp16 A operands, two tiles per K step
            h8 Ast[NKS];
            static_for<0, NKS>([&](auto pi) {
                constexpr int p = decltype(pi)::value;
                const h4 a = cvt4(acc[2 * p]);
                const h4 b = (2 * p + 1 < NT) ? cvt4(acc[(2 * p + 1) < NT ? 2 * p + 1 : 0])
                                              : h4{0, 0, 0, 0};
                Ast[p] = cat(a, b);
            });
            // Q^T fragments of this wave's row tile (for the in-chunk block and G)
            const int tokW = 16 * W + r16;
            const h8 QB0 = ld8(sm.qrow + tokW * RS + 8 * h);
            const h8 QB1 = ld8(sm.qrow + tokW * RS + 32 + 8 * h);

#pragma unroll
            for (int rt = 0; rt < 4; ++rt) {
                const int tok = 16 * rt + r16;
                h4 myl[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) myl[u] = ld4(sm.qrow + tok * RS + 16 * u + 4 * h);
                const h8 qa = ld8(sm.qperm + tok * RS + 16 * W);
                const h8 qb = ld8(sm.qperm + tok * RS + 16 * W + 8);
                const _Float16 qm[16] = {qa[0], qa[1], qa[2], qa[3], qa[4], qa[5], qa[6], qa[7],
                                         qb[0], qb[1], qb[2], qb[3], qb[4], qb[5], qb[6], qb[7]};
                f4 F0 = {0.f, 0.f, 0.f, 0.f}, F1 = {0.f, 0.f, 0.f, 0.f};
                auto gen = [&](auto ti) -> h4 {
                    constexpr int t = decltype(ti)::value;
                    constexpr Tile T = tile_of(W, t < NT ? t : 0);
                    if constexpr (t >= NT) {
                        return h4{0, 0, 0, 0};
                    } else if constexpr (T.kind == 0) {
                        return myl[T.u];
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
                if (rt == W) {
                    // in-chunk tril block: S^T tiles (rows t, cols i), i in this row tile
                    float gi = 0.f;
                    h4 wh[4];
#pragma unroll
                    for (int tt = 0; tt <= W; ++tt) {
                        f4 S = {0.f, 0.f, 0.f, 0.f};
                        S = mfma(ld8(sm.krow + (16 * tt + r16) * RS + 8 * h), QB0, S);
                        S = mfma(ld8(sm.krow + (16 * tt + r16) * RS + 32 + 8 * h), QB1, S);
                        f4 w;
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            const float s = S[i];
                            float x = fmaf(0.5f * s, s, 1.0f + s);
                            if (tt == W && (4 * h + i) > r16) x = 0.0f;
                            w[i] = x;
                            gi += x;
                        }
                        wh[tt] = cvt4(w);
                    }
#pragma unroll
                    for (int pa = 0; pa <= W / 2; ++pa) {
                        const int a = 2 * pa, b = 2 * pa + 1;
                        const h4 va = ld4(sm.vT + r16 * RS + 16 * a + 4 * h);
                        const h4 vb = (b <= W) ? ld4(sm.vT + r16 * RS + 16 * b + 4 * h)
                                               : h4{0, 0, 0, 0};
                        const h4 wb = (b <= W) ? wh[b < 4 ? b : 0] : h4{0, 0, 0, 0};
                        F0 = mfma(cat(va, vb), cat(wh[a], wb), F0);
                    }
                    // G_i = n0 + q.y2 + 1/2 q^T Y3 q + in-chunk row sum
                    float gq = 0.f;
#pragma unroll
                    for (int cc = 0; cc < 4; ++cc) {
                        const float ys = ldexpf(2.0f, -gexp);
                        f4 T;
#pragma unroll
                        for (int i = 0; i < 4; ++i) T[i] = ys * sm.y2[16 * cc + 4 * h + i];
                        T = mfma(ld8(sm.y3h + (16 * cc + r16) * RS + 8 * h), QB0, T);
                        T = mfma(ld8(sm.y3h + (16 * cc + r16) * RS + 32 + 8 * h), QB1, T);
#pragma unroll
                        for (int i = 0; i < 4; ++i) gq = fmaf((float)myl[cc][i], T[i], gq);
                    }
                    float part = fmaf(0.5f * ldexpf(1.0f, gexp), gq, gi);
                    part += __shfl_xor(part, 16);
                    part += __shfl_xor(part, 32);
                    if (h == 0) sm.g[16 * W + r16] = (float)n0 + part;
                }
                const f4 Fs = F0 + F1;
                *(f4 *)(sm.fpart + (W * C + tok) * SL + 4 * h) = Fs;
            }
            // this chunk's sums of k^ (for y2) and of scaled v (for x1)
            {
                const int m = 16 * W + r16;
                const h8 a = ld8(sm.kT + m * RS + 16 * h);
                const h8 b = ld8(sm.kT + m * RS + 16 * h + 8);
                float s = 0.f;
#pragma unroll
                for (int i = 0; i < 8; ++i) s += (float)a[i] + (float)b[i];
                s += __shfl_xor(s, 16);
                s += __shfl_xor(s, 32);
                if (h == 0) sm.y2c[m] = s;
                if (W == 0) {
                    const h8 va = ld8(sm.vT + r16 * RS + 16 * h);
                    const h8 vb = ld8(sm.vT + r16 * RS + 16 * h + 8);
                    float sv = 0.f;
#pragma unroll
                    for (int i = 0; i < 8; ++i) sv += (float)va[i] + (float)vb[i];
                    sv += __shfl_xor(sv, 16);
                    sv += __shfl_xor(sv, 32);
                    if (h == 0) sm.x1c[r16] = sv;
                }
            }
        }
        __syncthreads();

        // ---- (R) combine partials, divide, store ------------------------------
        {
            const int tok = tid >> 2, cq = tid & 3;
            f4 F = *(const f4 *)(sm.x1 + 4 * cq);
#pragma unroll
            for (int w = 0; w < NW; ++w) F += *(const f4 *)(sm.fpart + (w * C + tok) * SL + 4 * cq);
            const float Gi = sm.g[tok];
            if (n0 + tok < N) {
                const float sc = oscale / Gi;
                uint32_t lo = (uint32_t)f32_to_bf16(F[0] * sc) |
                              ((uint32_t)f32_to_bf16(F[1] * sc) << 16);
                uint32_t hi = (uint32_t)f32_to_bf16(F[2] * sc) |
                              ((uint32_t)f32_to_bf16(F[3] * sc) << 16);
                *(uint2 *)(out + (size_t)(n0 + tok) * D + SL * sl + 4 * cq) = uint2{lo, hi};
                if (g && sl == 0 && cq == 0) g[n0 + tok] = Gi;
            }
        }

        // ---- (U) state update S += Phi(K)^T V, Y3 += K^T K ---------------------
        {
            h8 Ak[4][2], Akh[4][2];
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int s = 0; s < 2; ++s) {
                    Ak[u][s] = ld8(sm.kT + (16 * u + r16) * RS + 32 * s + 8 * h);
                    Akh[u][s] = cat(scale4(h4{Ak[u][s][0], Ak[u][s][1], Ak[u][s][2], Ak[u][s][3]},
                                           (_Float16)0.5f),
                                    scale4(h4{Ak[u][s][4], Ak[u][s][5], Ak[u][s][6], Ak[u][s][7]},
                                           (_Float16)0.5f));
                }
            h8 Vf[2];
#pragma unroll
            for (int s = 0; s < 2; ++s) Vf[s] = ld8(sm.vT + r16 * RS + 32 * s + 8 * h);
            // linear tile
#pragma unroll
            for (int s = 0; s < 2; ++s) acc[0] = mfma(Ak[W][s], Vf[s], acc[0]);
            // quadratic tiles
            static_for<0, 16>([&](auto ii) {
                constexpr int idx = decltype(ii)::value;
                constexpr int m = W + 4 * idx;
                constexpr int u0 = m / 16;
                constexpr int t0 = first_tile(W, idx);
#pragma unroll
                for (int s = 0; s < 2; ++s) {
                    const h8 km = ld8(sm.kT + m * RS + 32 * s + 8 * h);
                    const h8 Wm = km * Vf[s];
                    static_for<u0, 4>([&](auto ui) {
                        constexpr int u = decltype(ui)::value;
                        constexpr int t = t0 + (u - u0);
                        if constexpr (u == u0) acc[t] = mfma(Akh[u][s], Wm, acc[t]);
                        else acc[t] = mfma(Ak[u][s], Wm, acc[t]);
                    });
                }
            });
            // Y3 tiles
            const int ntok = n0 + nvalid;
            const int gnext = max(0, pow2_exponent(64.0f * (float)ntok));
            const float gs = ldexpf(1.0f, -gnext);
            static_for<0, NY>([&](auto ki) {
                constexpr int kk = decltype(ki)::value;
                constexpr int u = y3_u(W, kk), u2 = y3_u2(W, kk);
#pragma unroll
                for (int s = 0; s < 2; ++s) y3acc[kk] = mfma(Ak[u][s], Ak[u2][s], y3acc[kk]);
                // lane: column m = 16*u2 + r16, rows l = 16*u + 4h + i
                const int mcol = 16 * u2 + r16;
                h4 hv;
#pragma unroll
                for (int i = 0; i < 4; ++i) hv[i] = (_Float16)(y3acc[kk][i] * gs);
                *(h4 *)(sm.y3h + mcol * RS + 16 * u + 4 * h) = hv;       // Y3[m][l]
                if (u != u2) {
#pragma unroll
                    for (int i = 0; i < 4; ++i) sm.y3h[(16 * u + 4 * h + i) * RS + mcol] = hv[i];
                }
            });
            gexp = gnext;
        }
        __syncthreads();
    }
}

__global__ __launch_bounds__(NTH, 1) void fwd_causal_kernel(const bf16_t *__restrict__ q,
                                                            const bf16_t *__restrict__ k,
                                                            const bf16_t *__restrict__ v,
                                                            bf16_t *__restrict__ out,
                                                            float *__restrict__ g, int N, int BH)
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

    // max |v| over this slice -> power-of-two scale
    const int tid = threadIdx.x;
    float vmax = 0.f;
    for (int p = tid; p < 2 * N; p += NTH) {
        const int n = p >> 1, hh = p & 1;
        float x[8];
        bf16x8_to_f32(*(const uint4 *)(v + (size_t)n * D + SL * sl + 8 * hh), x);
#pragma unroll
        for (int i = 0; i < 8; ++i) vmax = fmaxf(vmax, fabsf(x[i]));
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) vmax = fmaxf(vmax, __shfl_xor(vmax, o));
    if ((tid & 63) == 0) sm.red[tid >> 6] = vmax;
    if (tid < D) { sm.y2[tid] = 0.f; sm.y2c[tid] = 0.f; }
    if (tid < SL) { sm.x1[tid] = 0.f; sm.x1c[tid] = 0.f; }
    for (int e = tid; e < D * RS; e += NTH) sm.y3h[e] = (_Float16)0.0f;
    __syncthreads();
    vmax = fmaxf(fmaxf(sm.red[0], sm.red[1]), fmaxf(sm.red[2], sm.red[3]));
    const int vexp = pow2_exponent(vmax * 63.0f * (float)N);

    switch (tid >> 6) {
    case 0: run_wave<0>(sm, q, k, v, out, g, N, sl, vexp); break;
    case 1: run_wave<1>(sm, q, k, v, out, g, N, sl, vexp); break;
    case 2: run_wave<2>(sm, q, k, v, out, g, N, sl, vexp); break;
    default: run_wave<3>(sm, q, k, v, out, g, N, sl, vexp); break;
    }
}

}  // namespace mfma_causal

size_t mfma_causal_smem_bytes() { return sizeof(mfma_causal::Smem); }

hipError_t mfma_causal_fwd(const void *q, const void *k, const void *v, void *out, float *g,
                           int BH, int N, hipStream_t st)
{
    using namespace mfma_causal;
    static_assert(sizeof(Smem) <= 160 * 1024, "LDS budget");
    const size_t smem = sizeof(Smem);
    hipError_t e = hipFuncSetAttribute((const void *)fwd_causal_kernel,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(fwd_causal_kernel, dim3(BH * NSL), dim3(NTH), smem, st, (const bf16_t *)q,
                       (const bf16_t *)k, (const bf16_t *)v, (bf16_t *)out, g, N, BH);
    return hipGetLastError();
}

}  // namespace fm

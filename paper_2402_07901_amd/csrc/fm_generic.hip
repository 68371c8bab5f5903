// Generic Fastmax kernels: float32 VALU arithmetic, the moment state of one
// column slice held in LDS, tokens processed in chunks of CH.  General in
// (D, p, causal, dtype); the entry points route the quadratic-term dropout
// calls here and every other call to the MFMA kernels.  Like the MFMA
// kernels, they are checked against the fp64 CPU oracle; they are not a
// reference for the MFMA kernels.
//
// Notation (Sec. 2.4): phi(k) = [1, k, (k_m k_l)_{m<=l}] are the key-side
// features, psi(q) = [1, q, (c_ml q_m q_l)_{m<=l}] with c_mm = 1/2 and
// c_ml = 1 (m < l) the query-side ones, so psi(q).phi(k) = f_p(q.k).  The
// moment state of a slice of value columns J is S[f][j] = sum_n phi_f(k^_n)
// v'_nj, v' = [v | 1] (the ones column yields G).  Causal rows use the
// chunk-exclusive prefix of S plus the in-chunk tril block.
//
// Quadratic-term dropout (Sec. 2.4, dropout paragraph; Fig. 2), p = 2 only:
// the kernels' DROP variants multiply each key token's quadratic features
// phi_t(k^_n) by its keep bit times 1/(1 - rate) wherever they enter (the
// moment states built from keys, the in-chunk weights, and the backward's
// key-side contractions).  The weight of a pair is then
// w_in = 1 + s + sum_{m<=l} c_ml q_m q_l k_m k_l b~_n(m,l) instead of f_2(s).
#include <hip/hip_runtime.h>

#include "fm_common.h"
#include "fm_internal.h"

namespace fm {
namespace generic {

constexpr int CH = 16;    // tokens per chunk
constexpr int NT = 256;   // threads per workgroup

// Dropout arguments: keep bits ([B*H][N][mask_words(D)] words) and the scale
// 1/(1 - rate) of a kept feature.  bits == nullptr in the plain kernels.
// wblk (causal forward only): the masked in-chunk weights of every chunk,
// [B*H][chunks][CH][CH], written once per head by drop_wblk_kernel and read
// by every column slice.
struct Drop {
    const uint32_t *bits;
    float inv;
    const float *wblk;
};

// Multiplier of quadratic feature t of the token whose bit row is `row`.
__device__ __forceinline__ float keep_mult(const uint32_t *row, int t, float inv)
{
    return (row[t >> 5] >> (t & 31)) & 1u ? inv : 0.0f;
}

// Bit row of token n0 of a head (the chunk's first row).
template <int D>
__device__ __forceinline__ const uint32_t *mask_rows(const Drop &dr, int head, int N, int n0)
{
    return dr.bits + ((size_t)head * N + n0) * mask_words(D);
}

// Copies the bit rows of the chunk starting at token n0 into LDS (rows past
// N are zero), so the kernels read every bit from LDS.  Callers synchronise.
template <int D>
__device__ __forceinline__ void stage_mask(uint32_t *mk, const Drop &dr, int head, int N, int n0)
{
    constexpr int NW = mask_words(D);
    const uint32_t *src = mask_rows<D>(dr, head, N, n0);
    const int nv = min(CH, N - n0) * NW;
    for (int e = threadIdx.x; e < CH * NW; e += NT) mk[e] = e < nv ? src[e] : 0u;
}

template <int D, bool P2> struct feat {
    static constexpr int P = n_features(D, P2 ? 2 : 1);
    static constexpr int NPAIR = P2 ? D * (D + 1) / 2 : 0;
};

// Feature table in LDS: phi_f(x) = x[fa[f]] * x[fb[f]], where every staged
// row carries x[D] = 1 (load_std writes it into the padding column): f = 0 is
// (D, D), the linear feature f = 1 + m is (m, D), the quadratic feature of
// the pair (m, l), m <= l, is (m, l) (m-major order).  Branch-free in the
// feature index.
template <int D, bool P2>
__device__ void build_features(uint8_t *fa, uint8_t *fb)
{
    constexpr int P = feat<D, P2>::P;
    for (int f = threadIdx.x; f < P; f += NT) {
        int a = D, b = D;
        if (f >= 1 && f <= D) {
            a = f - 1;
        } else if (f > D) {
            int m = 0, r = f - 1 - D;
            while (r >= D - m) { r -= D - m; ++m; }
            a = m;
            b = m + r;
        }
        fa[f] = (uint8_t)a;
        fb[f] = (uint8_t)b;
    }
}

// p = 1 features [1, x]: feature f of row x.
__device__ __forceinline__ float phi1(int f, const float *x)
{
    if (f == 0) return 1.0f;
    return x[f - 1];
}

// Query-side factor of feature (a, b): 1/2 on the diagonal pairs, else 1.
template <int D>
__device__ __forceinline__ float psi_coef(int a, int b)
{
    return (a == b && a < D) ? 0.5f : 1.0f;
}

// Loads `rows` token rows starting at token n0 of a head and standardises
// them (Sec. 2.2, Eqs. 6-7: population std, no epsilon) into dst (stride
// D + 1, float32), times `scale` (the score scale on the query side, else 1).
// Rows past N are zero.  Optionally writes 1/std.
template <int D, typename T>
__device__ void load_std(const T *src, int n0, int N, float *dst, float *rstd_out,
                         float scale = 1.0f)
{
    constexpr int DP = D + 1;
    for (int e = threadIdx.x; e < CH * D; e += NT) {
        int r = e / D, d = e % D;
        int n = n0 + r;
        dst[r * DP + d] = n < N ? io<T>::ld(src, (size_t)n * D + d) : 0.0f;
    }
    __syncthreads();
    {
        // 16 lanes per row (NT = 16 * CH): each holds D / 16 channels; sums
        // over the row by butterfly shuffles within the 16 lanes
        static_assert(NT == 16 * CH && D % 16 == 0, "16 lanes per row");
        constexpr int E = D / 16;
        const int r = threadIdx.x >> 4, l = threadIdx.x & 15;
        float *x = dst + r * DP;
        float xv[E];
        float s = 0.0f;
#pragma unroll
        for (int i = 0; i < E; ++i) {
            xv[i] = x[l + 16 * i];
            s += xv[i];
        }
#pragma unroll
        for (int o = 8; o >= 1; o >>= 1) s += __shfl_xor(s, o, 16);
        const float mu = s * (1.0f / D);
        float var = 0.0f;
#pragma unroll
        for (int i = 0; i < E; ++i) {
            xv[i] -= mu;
            var = fmaf(xv[i], xv[i], var);
        }
#pragma unroll
        for (int o = 8; o >= 1; o >>= 1) var += __shfl_xor(var, o, 16);
        if (n0 + r < N) {
            const float rs = rsqrtf(var * (1.0f / D));
#pragma unroll
            for (int i = 0; i < E; ++i) x[l + 16 * i] = xv[i] * (rs * scale);
            if (rstd_out && l == 0) rstd_out[r] = rs;
        } else if (rstd_out && l == 0) {
            rstd_out[r] = 0.0f;
        }
        if (l == 0) x[D] = 1.0f;   // the constant of the feature table
    }
    __syncthreads();
}

// S[f][j] += sum_{r < CH} phi_f(x_r) val[r][j], j < WS.  DROP: the
// quadratic features of row r < nvalid are multiplied by the keep bits of
// its row in mrow (the chunk's rows staged in LDS by stage_mask).
template <int D, bool P2, int WS, bool DROP = false>
__device__ void state_update(float *S, const float *x, const float *val, const uint8_t *fa,
                             const uint8_t *fb, const uint32_t *mrow = nullptr, int nvalid = 0,
                             float inv = 1.0f)
{
    constexpr int P = feat<D, P2>::P;
    constexpr int DP = D + 1;
    constexpr int NW = mask_words(D);
    for (int f = threadIdx.x; f < P; f += NT) {
        const int a = P2 ? fa[f] : 0, b = P2 ? fb[f] : 0;
        const bool quad = f > D;
        const int t = quad ? f - 1 - D : 0;
        float acc[WS];
#pragma unroll
        for (int j = 0; j < WS; ++j) acc[j] = 0.0f;
        for (int r = 0; r < CH; ++r) {
            float ph = P2 ? x[r * DP + a] * x[r * DP + b] : phi1(f, x + r * DP);
            if constexpr (DROP) {
                const float km = r < nvalid ? keep_mult(mrow + r * NW, t, inv) : 0.0f;
                ph *= quad ? km : 1.0f;
            }
#pragma unroll
            for (int j = 0; j < WS; ++j) acc[j] = fmaf(ph, val[r * WS + j], acc[j]);
        }
#pragma unroll
        for (int j = 0; j < WS; ++j) S[f * WS + j] += acc[j];
    }
}

// out[r][j] += sum_f psi_f(x_r) S[f][j]   (LDS atomics; out is CH x WS).
// DROP: x holds keys, whose quadratic features take their keep bits.  At p = 2
// with slices of at most 3 columns (D = 128) a thread takes RPT = 4 rows, so
// each state row and table entry it reads serves four rows (measured slower
// for the wider slices of D <= 64).
template <int D, bool P2, int WS, bool DROP = false>
__device__ void contract_psi(const float *S, const float *x, float *out, const uint8_t *fa,
                             const uint8_t *fb, const uint32_t *mrow = nullptr, int nvalid = 0,
                             float inv = 1.0f)
{
    constexpr int P = feat<D, P2>::P;
    constexpr int DP = D + 1;
    constexpr int NW = mask_words(D);
    constexpr int RPT = (P2 && WS <= 3) ? 4 : 1;    // rows per thread
    constexpr int RG = CH / RPT;                     // row groups: rows rg + RG u
    constexpr int NG = NT / RG;                      // feature groups
    const int rg = threadIdx.x % RG, fg = threadIdx.x / RG;
    float acc[RPT][WS];
#pragma unroll
    for (int u = 0; u < RPT; ++u)
#pragma unroll
        for (int j = 0; j < WS; ++j) acc[u][j] = 0.0f;
    // p = 2 with one row per thread: unrolled so several table reads are in flight
    constexpr int UNROLL = P2 && RPT == 1 ? 4 : 1;
#pragma unroll UNROLL
    for (int f = fg; f < P; f += NG) {
        const int a = P2 ? fa[f] : 0, b = P2 ? fb[f] : 0;
        const bool quad = f > D;
        const float c = P2 ? psi_coef<D>(a, b) : 1.0f;
        float sv[WS];
#pragma unroll
        for (int j = 0; j < WS; ++j) sv[j] = S[f * WS + j];
#pragma unroll
        for (int u = 0; u < RPT; ++u) {
            const int r = rg + RG * u;
            const float *xr = x + r * DP;
            float ps = P2 ? c * (xr[a] * xr[b]) : phi1(f, xr);
            if constexpr (DROP) {
                const float km =
                    r < nvalid ? keep_mult(mrow + r * NW, quad ? f - 1 - D : 0, inv) : 0.0f;
                ps *= quad ? km : 1.0f;
            }
#pragma unroll
            for (int j = 0; j < WS; ++j) acc[u][j] = fmaf(ps, sv[j], acc[u][j]);
        }
    }
#pragma unroll
    for (int u = 0; u < RPT; ++u)
#pragma unroll
        for (int j = 0; j < WS; ++j) atomicAdd(&out[(rg + RG * u) * WS + j], acc[u][j]);
}

// Gradient-side contraction (backward):
//   out[r][a] = sum_{j<WS} coef[r][j] (S[1+a][j] + [p=2] sum_m x_rm S[(a,m)][j])
// which is the moment form of sum_n f'(s_rn) (coef_r . val_n) y_n[a] when S
// holds the moments of (y, val).  DROP: x holds keys, and x_rm carries the
// keep multiplier of row r's feature (a, m).
template <int D, bool P2, int WS, bool DROP = false>
__device__ void contract_grad(const float *S, const float *x, const float *coef, float *out,
                              const uint32_t *mrow = nullptr, int nvalid = 0, float inv = 1.0f)
{
    constexpr int DP = D + 1;
    constexpr int AG = NT / CH;          // a-groups
    constexpr int NW = mask_words(D);
    const int r = threadIdx.x % CH, ag = threadIdx.x / CH;
    const float *xr = x + r * DP;
    // (a, m) outer, the WS columns inner: each state row and (DROP) each keep
    // bit is read once for all columns
    const uint32_t *row = DROP ? mrow + (r < nvalid ? r : 0) * NW : nullptr;
    for (int a = ag; a < D; a += AG) {
        float inner[WS];
#pragma unroll
        for (int j = 0; j < WS; ++j) inner[j] = S[(1 + a) * WS + j];
        if constexpr (P2) {
            // packed index of the pair (min(a, m), max(a, m)), walked with adds:
            // t(m, a) = t(m, m) + a - m for m < a, t(a, m) = t(a, a) + m - a
            const int taa = a * D - a * (a - 1) / 2;
            int tmm = 0;
            for (int m = 0; m < D; ++m) {
                const int pf = 1 + D + (m < a ? tmm + a - m : taa + m - a);
                tmm += D - m;
                float xm = xr[m];
                if constexpr (DROP)
                    xm = r < nvalid ? xm * keep_mult(row, pf - 1 - D, inv) : 0.0f;
#pragma unroll
                for (int j = 0; j < WS; ++j) inner[j] = fmaf(xm, S[pf * WS + j], inner[j]);
            }
        }
        float acc = 0.0f;
#pragma unroll
        for (int j = 0; j < WS; ++j) acc = fmaf(coef[r * WS + j], inner[j], acc);
        out[r * D + a] = acc;
    }
}

// Dropout weight of one (query, key) pair, xq already scaled by the score
// scale: 1 + s + sum_{m<=l} c_ml z_m z_l b~_t(m,l), z = xq (.) xk, c_mm = 1/2.
template <int D>
__device__ float drop_weight(const float *xq, const float *xk, const uint32_t *row, float inv)
{
    float s = 0.0f, quad = 0.0f;
    int t = 0;
    uint32_t word = 0;
    for (int m = 0; m < D; ++m) {
        const float zm = xq[m] * xk[m];
        s += zm;
        float inner = 0.0f;
        for (int l = m; l < D; ++l, ++t) {
            if ((t & 31) == 0) word = row[t >> 5];
            const float zl = l == m ? 0.5f * zm : xq[l] * xk[l];
            if ((word >> (t & 31)) & 1u) inner += zl;
        }
        quad = fmaf(zm, inner, quad);
    }
    return 1.0f + s + quad * inv;
}

// d w / d xq_a = xk_a h_a and d w / d xk_a = xq_a h_a for the dropout weight,
// h_a = 1 + sum_l xq_l xk_l b~_t(a,l).
// One loop over l (the lanes of a wave hold different a, so split loops would
// run both to their longest): feature (l, a), l < a, is t(l, l) + a - l with
// t(l + 1, l + 1) = t(l, l) + D - l; feature (a, l), l >= a, is t(a, a) + l - a.
template <int D>
__device__ float drop_h(const float *xq, const float *xk, const uint32_t *row, int a, float inv)
{
    float acc = 0.0f;
    const int taa = a * D - a * (a - 1) / 2;   // t(a, a)
    int tll = 0;                               // t(l, l)
    for (int l = 0; l < D; ++l) {
        const int t = l < a ? tll + a - l : taa + l - a;
        if ((row[t >> 5] >> (t & 31)) & 1u) acc = fmaf(xq[l], xk[l], acc);
        tll += D - l;
    }
    return fmaf(acc, inv, 1.0f);
}

// Masked in-chunk weights of the causal forward, once per (head, chunk):
// out[i][t] = w_it for t <= i < rows left, else 0.  grid = (B*H, y, z), chunk
// y + 65535 z (grid y is at most 65535).
template <int D, typename T>
__global__ __launch_bounds__(NT) void drop_wblk_kernel(const T *__restrict__ q,
                                                       const T *__restrict__ k,
                                                       float *__restrict__ wblk, int N,
                                                       float qs, Drop dr)
{
    constexpr int DP = D + 1;
    __shared__ float xq[CH * DP];
    __shared__ float xk[CH * DP];
    __shared__ uint32_t mk[CH * mask_words(D)];
    const int head = blockIdx.x, nch = (N + CH - 1) / CH;
    const int c = blockIdx.y + 65535 * blockIdx.z, n0 = c * CH;
    if (c >= nch) return;   // the whole block, before any barrier
    const size_t hb = (size_t)head * N * D;
    stage_mask<D>(mk, dr, head, N, n0);
    load_std<D>(q + hb, n0, N, xq, nullptr, qs);   // synchronises the staging too
    load_std<D>(k + hb, n0, N, xk, nullptr);
    const int i = threadIdx.x / CH, t = threadIdx.x % CH;
    float w = 0.0f;
    // keys past N are never seen by a valid row (t <= i < N)
    if (t <= i && n0 + i < N)
        w = drop_weight<D>(xq + i * DP, xk + t * DP, mk + t * mask_words(D), dr.inv);
    wblk[((size_t)head * nch + c) * (CH * CH) + threadIdx.x] = w;
}

// ---------------------------------------------------------------------------
// Forward.  grid = (B*H, slices, segments); slice s owns value columns
// [s*W, s*W+W) plus the ones column (local index W), so every slice has G for
// its divide.  With several segments (few heads), seg_state_kernel first
// writes each segment's moment contribution to sseg; a causal segment starts
// its scan from the sum of the earlier segments (the exclusive prefix of
// Sec. 2.4's causal moments at the segment start), a non-causal one contracts
// its queries against the sum of all segments.
// ---------------------------------------------------------------------------
template <int D, bool P2, int WS, typename T, bool DROP = false>
__global__ __launch_bounds__(NT) void seg_state_kernel(const T *__restrict__ k,
                                                       const T *__restrict__ v,
                                                       float *__restrict__ sseg, int N, int cps,
                                                       Drop dr = Drop{nullptr, 1.0f, nullptr})
{
    constexpr int P = feat<D, P2>::P;
    constexpr int W = WS - 1;
    constexpr int DP = D + 1;

    __shared__ float S[P * WS];
    __shared__ float xk[CH * DP];
    __shared__ float vv[CH * WS];
    __shared__ uint8_t fa[P];
    __shared__ uint8_t fb[P];
    __shared__ uint32_t mk[DROP ? CH * mask_words(D) : 1];

    const int head = blockIdx.x, c0 = blockIdx.y * W, seg = blockIdx.z;
    const size_t hb = (size_t)head * N * D;
    k += hb;
    v += hb;
    for (int e = threadIdx.x; e < P * WS; e += NT) S[e] = 0.0f;
    build_features<D, P2>(fa, fb);
    __syncthreads();
    const int nch = (N + CH - 1) / CH;
    const int cb = seg * cps, ce = min(nch, cb + cps);
    for (int c = cb; c < ce; ++c) {
        load_std<D>(k, c * CH, N, xk, nullptr);
        for (int e = threadIdx.x; e < CH * WS; e += NT) {
            int r = e / WS, j = e % WS, n = c * CH + r;
            float x = 0.0f;
            if (n < N) {
                if (j == W) x = 1.0f;
                else if (c0 + j < D) x = io<T>::ld(v, (size_t)n * D + c0 + j);
            }
            vv[e] = x;
        }
        if constexpr (DROP) stage_mask<D>(mk, dr, head, N, c * CH);
        __syncthreads();
        if constexpr (DROP)
            state_update<D, P2, WS, true>(S, xk, vv, fa, fb, mk, CH, dr.inv);
        else
            state_update<D, P2, WS>(S, xk, vv, fa, fb);
        __syncthreads();
    }
    float *dst = sseg + (((size_t)head * gridDim.y + blockIdx.y) * gridDim.z + seg) * P * WS;
    for (int e = threadIdx.x; e < P * WS; e += NT) dst[e] = S[e];
}

// In place over the segments of each (head, slice): causal -> the exclusive
// prefix sum (segment s gets the sum of segments < s; with REVERSE the
// exclusive suffix, the sum of segments > s), non-causal -> the total in
// segment 0.  One thread per state element.
template <int PWS, bool CAUSAL, bool REVERSE = false>
__global__ __launch_bounds__(NT) void seg_prefix_kernel(float *__restrict__ sseg, int nseg)
{
    const int e = blockIdx.x * NT + threadIdx.x;
    if (e >= PWS) return;
    float *base = sseg + (size_t)blockIdx.y * nseg * PWS + e;
    float run = 0.0f;
    // eight segments loaded before any is overwritten: the loads are in
    // flight together instead of one round trip each
    constexpr int U = 8;
    for (int s0 = 0; s0 < nseg; s0 += U) {
        float x[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int sg = REVERSE ? nseg - 1 - (s0 + u) : s0 + u;
            x[u] = s0 + u < nseg ? base[(size_t)sg * PWS] : 0.0f;
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int sg = REVERSE ? nseg - 1 - (s0 + u) : s0 + u;
            if (CAUSAL && s0 + u < nseg) base[(size_t)sg * PWS] = run;
            run += x[u];
        }
    }
    if (!CAUSAL) base[0] = run;
}

template <int D, bool P2, int WS, bool CAUSAL, typename T, bool DROP = false>
__global__ __launch_bounds__(NT) void fwd_kernel(const T *__restrict__ q, const T *__restrict__ k,
                                                 const T *__restrict__ v, T *__restrict__ out,
                                                 float *__restrict__ g, int N, int cps,
                                                 const float *__restrict__ sseg, float qs,
                                                 Drop dr = Drop{nullptr, 1.0f, nullptr})
{
    constexpr int P = feat<D, P2>::P;
    constexpr int W = WS - 1;
    constexpr int DP = D + 1;
    constexpr int POW = P2 ? 2 : 1;

    __shared__ float S[P * WS];
    __shared__ float xq[CH * DP];
    __shared__ float xk[CH * DP];
    __shared__ float vv[CH * WS];
    __shared__ float wblk[CH * CH];
    __shared__ float F[CH * WS];
    __shared__ uint8_t fa[P];
    __shared__ uint8_t fb[P];
    __shared__ uint32_t mk[DROP ? CH * mask_words(D) : 1];

    const int head = blockIdx.x;
    const int c0 = blockIdx.y * W;
    const size_t hb = (size_t)head * N * D;
    q += hb;
    k += hb;
    v += hb;
    out += hb;
    if (g) g += (size_t)head * N;

    const int nseg = gridDim.z, seg = blockIdx.z;
    {
        // initial state: the sum of the earlier segments (causal) or of all
        // of them, as seg_prefix_kernel left it in this segment's slot (in
        // segment 0's for non-causal)
        const float *src = sseg ? sseg + (((size_t)head * gridDim.y + blockIdx.y) * nseg +
                                          (CAUSAL ? seg : 0)) * P * WS
                                : nullptr;
        for (int e = threadIdx.x; e < P * WS; e += NT) S[e] = src ? src[e] : 0.0f;
    }
    build_features<D, P2>(fa, fb);
    __syncthreads();

    auto load_vals = [&](int n0) {
        for (int e = threadIdx.x; e < CH * WS; e += NT) {
            int r = e / WS, j = e % WS, n = n0 + r;
            float x = 0.0f;
            if (n < N) {
                if (j == W) x = 1.0f;
                else if (c0 + j < D) x = io<T>::ld(v, (size_t)n * D + c0 + j);
            }
            vv[e] = x;
        }
    };
    auto write_out = [&](int n0) {
        for (int e = threadIdx.x; e < CH * W; e += NT) {
            int r = e / W, j = e % W, n = n0 + r;
            if (n < N && c0 + j < D)
                io<T>::st(out, (size_t)n * D + c0 + j, F[r * WS + j] / F[r * WS + W]);
        }
        if (g && blockIdx.y == 0)
            for (int r = threadIdx.x; r < CH; r += NT)
                if (n0 + r < N) g[n0 + r] = F[r * WS + W];
    };

    const int nch = (N + CH - 1) / CH;
    const int cb = seg * cps, ce = min(nch, cb + cps);
    if (!CAUSAL) {
        if (!sseg) {
            for (int c = 0; c < nch; ++c) {
                load_std<D>(k, c * CH, N, xk, nullptr);
                load_vals(c * CH);
                if constexpr (DROP) stage_mask<D>(mk, dr, head, N, c * CH);
                __syncthreads();
                if constexpr (DROP)
                    state_update<D, P2, WS, true>(S, xk, vv, fa, fb, mk, CH, dr.inv);
                else
                    state_update<D, P2, WS>(S, xk, vv, fa, fb);
                __syncthreads();
            }
        }
        for (int c = cb; c < ce; ++c) {
            load_std<D>(q, c * CH, N, xq, nullptr, qs);
            for (int e = threadIdx.x; e < CH * WS; e += NT) F[e] = 0.0f;
            __syncthreads();
            contract_psi<D, P2, WS>(S, xq, F, fa, fb);
            __syncthreads();
            write_out(c * CH);
            __syncthreads();
        }
    } else {
        for (int c = cb; c < ce; ++c) {
            const int n0 = c * CH;
            load_std<D>(q, n0, N, xq, nullptr, qs);
            load_std<D>(k, n0, N, xk, nullptr);
            load_vals(n0);
            if constexpr (DROP) stage_mask<D>(mk, dr, head, N, n0);
            // in-chunk tril block of weights
            {
                int i = threadIdx.x / CH, t = threadIdx.x % CH;
                float w = 0.0f;
                if constexpr (DROP) {
                    w = dr.wblk[((size_t)head * nch + c) * (CH * CH) + i * CH + t];
                } else if (t <= i) {
                    float s = 0.0f;
                    for (int d = 0; d < D; ++d) s = fmaf(xq[i * DP + d], xk[t * DP + d], s);
                    w = taylor<POW>(s);
                }
                wblk[i * CH + t] = w;
            }
            __syncthreads();
            for (int e = threadIdx.x; e < CH * WS; e += NT) {
                int i = e / WS, j = e % WS;
                float acc = 0.0f;
                for (int t = 0; t <= i; ++t) acc = fmaf(wblk[i * CH + t], vv[t * WS + j], acc);
                F[e] = acc;
            }
            __syncthreads();
            contract_psi<D, P2, WS>(S, xq, F, fa, fb);   // exclusive prefix S_<c
            __syncthreads();
            write_out(n0);
            if constexpr (DROP)
                state_update<D, P2, WS, true>(S, xk, vv, fa, fb, mk, CH, dr.inv);
            else
                state_update<D, P2, WS>(S, xk, vv, fa, fb);
            __syncthreads();
        }
    }
}

// ---------------------------------------------------------------------------
// Backward.
//   u_i = dO_i / G_i,  c_i = (dO_i . O_i) / G_i,  u~_i = [u_i, -c_i]
//   dw_in = u~_i . v'_n,  ds_in = f'(s_in) dw_in       (Sec. 2.3, Eq. bound)
//   dq^_i = sum_n ds_in k^_n,  dk^_n = sum_i ds_in q^_i,  dv_n = sum_i w_in u_i
// Columns j run over the D+1 columns of v' / u~; slices split them.
// ---------------------------------------------------------------------------

// c_i = (dO_i . O_i) / G_i, one row per thread.
template <int D, typename T>
__global__ __launch_bounds__(NT) void bwd_rowdot_kernel(const T *__restrict__ o,
                                                        const T *__restrict__ dout,
                                                        const float *__restrict__ g,
                                                        float *__restrict__ cvec, size_t rows)
{
    size_t r = (size_t)blockIdx.x * NT + threadIdx.x;
    if (r >= rows) return;
    float acc = 0.0f;
    for (int d = 0; d < D; ++d)
        acc = fmaf(io<T>::ld(dout, r * D + d), io<T>::ld(o, r * D + d), acc);
    cvec[r] = acc / g[r];
}

// Loads CH rows of u~ restricted to global columns [gc0, gc0 + WS).
template <int D, int WS, typename T>
__device__ void load_utilde(const T *dout, const float *g, const float *cvec, int n0, int N,
                            int gc0, float *dst)
{
    for (int e = threadIdx.x; e < CH * WS; e += NT) {
        int r = e / WS, j = e % WS, n = n0 + r, gc = gc0 + j;
        float x = 0.0f;
        if (n < N) {
            if (gc < D) x = io<T>::ld(dout, (size_t)n * D + gc) / g[n];
            else if (gc == D) x = -cvec[n];
        }
        dst[e] = x;
    }
}

template <int D, int WS, typename T>
__device__ void load_vprime(const T *v, int n0, int N, int gc0, float *dst)
{
    for (int e = threadIdx.x; e < CH * WS; e += NT) {
        int r = e / WS, j = e % WS, n = n0 + r, gc = gc0 + j;
        float x = 0.0f;
        if (n < N) {
            if (gc < D) x = io<T>::ld(v, (size_t)n * D + gc);
            else if (gc == D) x = 1.0f;
        }
        dst[e] = x;
    }
}

// In-chunk (tril) part of all three gradients; plain stores initialise the
// float32 accumulators (zeros for the non-causal problem, whose every pair is
// handled by the moment kernels).
// DROP: E holds dw alone and Wm the dropout weight; the derivative factor
// is the per-channel h of drop_h, with the key rows' keep bits staged in LDS.
template <int D, bool P2, bool CAUSAL, typename T, bool DROP = false>
__global__ __launch_bounds__(NT) void bwd_intra_kernel(
    const T *__restrict__ q, const T *__restrict__ k, const T *__restrict__ v,
    const T *__restrict__ dout, const float *__restrict__ g, const float *__restrict__ cvec,
    float *__restrict__ dqh, float *__restrict__ dkh, float *__restrict__ dva, int N, float qs,
    Drop dr = Drop{nullptr, 1.0f, nullptr})
{
    constexpr int DP = D + 1;
    constexpr int D1 = D + 1;
    constexpr int POW = P2 ? 2 : 1;
    constexpr int NW = mask_words(D);
    __shared__ float xq[CH * DP];
    __shared__ float xk[CH * DP];
    __shared__ float vp[CH * D1];
    __shared__ float ut[CH * D1];
    __shared__ float E[CH * CH];   // f'(s) dw
    __shared__ float Wm[CH * CH];  // f(s)
    __shared__ uint32_t mk[DROP ? CH * NW : 1];
    __shared__ float accq[DROP ? CH * D : 1];   // DROP: in-chunk dq^, dk^ sums
    __shared__ float acck[DROP ? CH * D : 1];

    // chunk y + 65535 z (grid y is at most 65535); blocks past the last chunk
    // leave before any barrier
    const int head = blockIdx.x, c = blockIdx.y + 65535 * blockIdx.z, n0 = c * CH;
    if (n0 >= N) return;
    const size_t hb = (size_t)head * N * D;
    q += hb; k += hb; v += hb; dout += hb;
    g += (size_t)head * N;
    cvec += (size_t)head * N;
    dqh += hb; dkh += hb; dva += hb;

    if (!CAUSAL) {
        for (int e = threadIdx.x; e < CH * D; e += NT) {
            int r = e / D, n = n0 + r;
            if (n < N) {
                size_t o = (size_t)n * D + e % D;
                dqh[o] = 0.0f; dkh[o] = 0.0f; dva[o] = 0.0f;
            }
        }
        return;
    }
    load_std<D>(q, n0, N, xq, nullptr, qs);
    load_std<D>(k, n0, N, xk, nullptr);
    load_vprime<D, D1>(v, n0, N, 0, vp);
    load_utilde<D, D1>(dout, g, cvec, n0, N, 0, ut);
    if constexpr (DROP) {
        stage_mask<D>(mk, dr, head, N, n0);
        for (int e = threadIdx.x; e < CH * D; e += NT) accq[e] = acck[e] = 0.0f;
    }
    __syncthreads();
    {
        int i = threadIdx.x / CH, t = threadIdx.x % CH;
        float e = 0.0f, w = 0.0f;
        if (t <= i && n0 + i < N) {
            float dw = 0.0f;
            for (int j = 0; j < D1; ++j) dw = fmaf(ut[i * D1 + j], vp[t * D1 + j], dw);
            if constexpr (DROP) {
                e = dw;
                w = drop_weight<D>(xq + i * DP, xk + t * DP, mk + t * NW, dr.inv);
            } else {
                float s = 0.0f;
                for (int d = 0; d < D; ++d) s = fmaf(xq[i * DP + d], xk[t * DP + d], s);
                e = dtaylor<POW>(s) * dw;
                w = taylor<POW>(s);
            }
        }
        E[i * CH + t] = e;
        Wm[i * CH + t] = w;
    }
    __syncthreads();
    if constexpr (DROP) {
        // one (pair, channel) per item: h of the pair (i, t), t <= i, is
        // shared by dq^_i (k_t h) and dk^_t (q_i h)
        constexpr int NPR = CH * (CH + 1) / 2;
        for (int e = threadIdx.x; e < NPR * D; e += NT) {
            const int pr = e / D, a = e % D;
            int i = 0;
            while ((i + 1) * (i + 2) / 2 <= pr) ++i;
            const int t = pr - i * (i + 1) / 2;
            const float eit = E[i * CH + t];   // 0 for rows past N
            if (eit == 0.0f) continue;
            const float h = drop_h<D>(xq + i * DP, xk + t * DP, mk + t * NW, a, dr.inv);
            atomicAdd(&accq[i * D + a], eit * xk[t * DP + a] * h);
            atomicAdd(&acck[t * D + a], eit * xq[i * DP + a] * h);
        }
        __syncthreads();
    }
    for (int e = threadIdx.x; e < CH * D; e += NT) {
        int r = e / D, a = e % D, n = n0 + r;
        if (n >= N) continue;
        float aq = 0.0f, ak = 0.0f, av = 0.0f;
        if constexpr (DROP) {
            aq = accq[r * D + a];
            ak = acck[r * D + a];
            for (int t = 0; t < CH; ++t) av = fmaf(Wm[t * CH + r], ut[t * D1 + a], av);
        } else {
            for (int t = 0; t < CH; ++t) {
                aq = fmaf(E[r * CH + t], xk[t * DP + a], aq);   // row r as query
                ak = fmaf(E[t * CH + r], xq[t * DP + a], ak);   // row r as key
                av = fmaf(Wm[t * CH + r], ut[t * D1 + a], av);
            }
        }
        size_t o = (size_t)n * D + a;
        dqh[o] = aq;
        dkh[o] = ak;
        dva[o] = av;
    }
}

// dq^ from the forward-direction moments of (k^, v'): grid = (B*H, slices over
// the D+1 columns of v').  Causal rows see the chunk-exclusive prefix.
template <int D, bool P2, int WS, bool CAUSAL, typename T, bool DROP = false>
__global__ __launch_bounds__(NT) void bwd_qscan_kernel(
    const T *__restrict__ q, const T *__restrict__ k, const T *__restrict__ v,
    const T *__restrict__ dout, const float *__restrict__ g, const float *__restrict__ cvec,
    float *__restrict__ dqh, int N, float qs, const float *__restrict__ sseg, int cps,
    Drop dr = Drop{nullptr, 1.0f, nullptr})
{
    constexpr int P = feat<D, P2>::P;
    constexpr int DP = D + 1;
    __shared__ float S[P * WS];
    __shared__ float xq[CH * DP];
    __shared__ float xk[CH * DP];
    __shared__ float vp[CH * WS];
    __shared__ float ut[CH * WS];
    __shared__ float part[CH * D];
    __shared__ uint8_t fa[P];
    __shared__ uint8_t fb[P];
    __shared__ uint32_t mk[DROP ? CH * mask_words(D) : 1];

    const int head = blockIdx.x, gc0 = blockIdx.y * WS;
    const size_t hb = (size_t)head * N * D;
    q += hb; k += hb; v += hb; dout += hb; dqh += hb;
    g += (size_t)head * N;
    cvec += (size_t)head * N;

    // initial state: the moments of the earlier segments (causal) or of all
    // of them, as seg_prefix_kernel left them (zero with one segment)
    const int nseg = gridDim.z, seg = blockIdx.z;
    {
        const float *src = sseg ? sseg + (((size_t)head * gridDim.y + blockIdx.y) * nseg +
                                          (CAUSAL ? seg : 0)) * P * WS
                                : nullptr;
        for (int e = threadIdx.x; e < P * WS; e += NT) S[e] = src ? src[e] : 0.0f;
    }
    build_features<D, P2>(fa, fb);
    __syncthreads();
    const int nch = (N + CH - 1) / CH;
    const int cb = seg * cps, ce = min(nch, cb + cps);

    auto contract_and_add = [&](int n0) {
        load_std<D>(q, n0, N, xq, nullptr, qs);
        load_utilde<D, WS>(dout, g, cvec, n0, N, gc0, ut);
        __syncthreads();
        contract_grad<D, P2, WS>(S, xq, ut, part);
        __syncthreads();
        for (int e = threadIdx.x; e < CH * D; e += NT) {
            int n = n0 + e / D;
            if (n < N) atomicAdd(&dqh[(size_t)n * D + e % D], part[e]);
        }
        __syncthreads();
    };
    auto update = [&](int n0) {
        load_std<D>(k, n0, N, xk, nullptr);
        load_vprime<D, WS>(v, n0, N, gc0, vp);
        if constexpr (DROP) stage_mask<D>(mk, dr, head, N, n0);
        __syncthreads();
        if constexpr (DROP)
            state_update<D, P2, WS, true>(S, xk, vp, fa, fb, mk, CH, dr.inv);
        else
            state_update<D, P2, WS>(S, xk, vp, fa, fb);
        __syncthreads();
    };
    if (!CAUSAL) {
        if (!sseg)
            for (int c = 0; c < nch; ++c) update(c * CH);
        for (int c = cb; c < ce; ++c) contract_and_add(c * CH);
    } else {
        for (int c = cb; c < ce; ++c) {
            contract_and_add(c * CH);
            update(c * CH);
        }
    }
}

// dk^ and dv from the reverse-direction moments of (q^, u~):
//   T[f][j] = sum_i phi_f(q^_i) u~_ij over rows i after the chunk (causal) or
//   all rows; dk^_n[a] += sum_j v'_nj (T[1+a][j] + sum_m k^_nm T[(a,m)][j]),
//   dv_n[j] += sum_f psi_f(k^_n) T[f][j].
template <int D, bool P2, int WS, bool CAUSAL, typename T, bool DROP = false>
__global__ __launch_bounds__(NT) void bwd_kscan_kernel(
    const T *__restrict__ q, const T *__restrict__ k, const T *__restrict__ v,
    const T *__restrict__ dout, const float *__restrict__ g, const float *__restrict__ cvec,
    float *__restrict__ dkh, float *__restrict__ dva, int N, float qs,
    const float *__restrict__ sseg, int cps, Drop dr = Drop{nullptr, 1.0f, nullptr})
{
    constexpr int P = feat<D, P2>::P;
    constexpr int DP = D + 1;
    __shared__ float S[P * WS];
    __shared__ float xq[CH * DP];
    __shared__ float xk[CH * DP];
    __shared__ float vp[CH * WS];
    __shared__ float ut[CH * WS];
    __shared__ float part[CH * D];
    __shared__ float pv[CH * WS];
    __shared__ uint8_t fa[P];
    __shared__ uint8_t fb[P];
    __shared__ uint32_t mk[DROP ? CH * mask_words(D) : 1];

    const int head = blockIdx.x, gc0 = blockIdx.y * WS;
    const size_t hb = (size_t)head * N * D;
    q += hb; k += hb; v += hb; dout += hb; dkh += hb; dva += hb;
    g += (size_t)head * N;
    cvec += (size_t)head * N;

    // initial state: the moments of the later segments (causal: exclusive
    // suffix) or of all of them (zero with one segment)
    const int nseg = gridDim.z, seg = blockIdx.z;
    {
        const float *src = sseg ? sseg + (((size_t)head * gridDim.y + blockIdx.y) * nseg +
                                          (CAUSAL ? seg : 0)) * P * WS
                                : nullptr;
        for (int e = threadIdx.x; e < P * WS; e += NT) S[e] = src ? src[e] : 0.0f;
    }
    build_features<D, P2>(fa, fb);
    __syncthreads();
    const int nch = (N + CH - 1) / CH;
    const int cb = seg * cps, ce = min(nch, cb + cps);

    auto contract_and_add = [&](int n0) {
        load_std<D>(k, n0, N, xk, nullptr);
        load_vprime<D, WS>(v, n0, N, gc0, vp);
        for (int e = threadIdx.x; e < CH * WS; e += NT) pv[e] = 0.0f;
        if constexpr (DROP) stage_mask<D>(mk, dr, head, N, n0);
        __syncthreads();
        if constexpr (DROP) {
            contract_grad<D, P2, WS, true>(S, xk, vp, part, mk, CH, dr.inv);
            contract_psi<D, P2, WS, true>(S, xk, pv, fa, fb, mk, CH, dr.inv);
        } else {
            contract_grad<D, P2, WS>(S, xk, vp, part);
            contract_psi<D, P2, WS>(S, xk, pv, fa, fb);
        }
        __syncthreads();
        for (int e = threadIdx.x; e < CH * D; e += NT) {
            int n = n0 + e / D;
            if (n < N) atomicAdd(&dkh[(size_t)n * D + e % D], part[e]);
        }
        for (int e = threadIdx.x; e < CH * WS; e += NT) {
            int n = n0 + e / WS, gc = gc0 + e % WS;
            if (n < N && gc < D) atomicAdd(&dva[(size_t)n * D + gc], pv[e]);
        }
        __syncthreads();
    };
    auto update = [&](int n0) {
        load_std<D>(q, n0, N, xq, nullptr, qs);
        load_utilde<D, WS>(dout, g, cvec, n0, N, gc0, ut);
        __syncthreads();
        state_update<D, P2, WS>(S, xq, ut, fa, fb);
        __syncthreads();
    };
    if (!CAUSAL) {
        if (!sseg)
            for (int c = 0; c < nch; ++c) update(c * CH);
        for (int c = cb; c < ce; ++c) contract_and_add(c * CH);
    } else {
        for (int c = ce - 1; c >= cb; --c) {
            contract_and_add(c * CH);
            update(c * CH);
        }
    }
}

// Moment sums of one segment of chunks for the backward scans (all segments
// in parallel): SIDE 0 -> sum phi(k^_n) v'_n (the q-scan's state), SIDE 1 ->
// sum phi(qs q^_i) u~_i (the k-scan's state), columns gc0.. of the D + 1.
template <int D, bool P2, int WS, int SIDE, typename T, bool DROP = false>
__global__ __launch_bounds__(NT) void bwd_seg_state_kernel(
    const T *__restrict__ q, const T *__restrict__ k, const T *__restrict__ v,
    const T *__restrict__ dout, const float *__restrict__ g, const float *__restrict__ cvec,
    float *__restrict__ sseg, int N, float qs, int cps, Drop dr = Drop{nullptr, 1.0f, nullptr})
{
    constexpr int P = feat<D, P2>::P;
    constexpr int DP = D + 1;
    __shared__ float S[P * WS];
    __shared__ float xs[CH * DP];
    __shared__ float vals[CH * WS];
    __shared__ uint8_t fa[P];
    __shared__ uint8_t fb[P];
    __shared__ uint32_t mk[DROP && SIDE == 0 ? CH * mask_words(D) : 1];

    const int head = blockIdx.x, gc0 = blockIdx.y * WS;
    const int nseg = gridDim.z, seg = blockIdx.z;
    const size_t hb = (size_t)head * N * D;
    q += hb; k += hb; v += hb; dout += hb;
    g += (size_t)head * N;
    cvec += (size_t)head * N;
    for (int e = threadIdx.x; e < P * WS; e += NT) S[e] = 0.0f;
    build_features<D, P2>(fa, fb);
    __syncthreads();
    const int nch = (N + CH - 1) / CH;
    const int cb = seg * cps, ce = min(nch, cb + cps);
    for (int c = cb; c < ce; ++c) {
        if constexpr (SIDE == 0) {
            load_std<D>(k, c * CH, N, xs, nullptr);
            load_vprime<D, WS>(v, c * CH, N, gc0, vals);
            if constexpr (DROP) stage_mask<D>(mk, dr, head, N, c * CH);
        } else {
            load_std<D>(q, c * CH, N, xs, nullptr, qs);
            load_utilde<D, WS>(dout, g, cvec, c * CH, N, gc0, vals);
        }
        __syncthreads();
        if constexpr (DROP && SIDE == 0)   // keys: their quadratic features are masked
            state_update<D, P2, WS, true>(S, xs, vals, fa, fb, mk, CH, dr.inv);
        else
            state_update<D, P2, WS>(S, xs, vals, fa, fb);
        __syncthreads();
    }
    float *dst = sseg + (((size_t)head * gridDim.y + blockIdx.y) * nseg + seg) * P * WS;
    for (int e = threadIdx.x; e < P * WS; e += NT) dst[e] = S[e];
}

// Back through Eqs. (6)-(7) and cast: dx = (dx^ - mean dx^ - x^ mean(dx^ x^)) / std.
template <int D, typename T>
__global__ __launch_bounds__(NT) void bwd_finish_kernel(
    const T *__restrict__ q, const T *__restrict__ k, const float *__restrict__ dqh,
    const float *__restrict__ dkh, const float *__restrict__ dva, T *__restrict__ dq,
    T *__restrict__ dk, T *__restrict__ dv, size_t rows, float qs)
{
    size_t r = (size_t)blockIdx.x * NT + threadIdx.x;
    if (r >= rows) return;
    const size_t b = r * D;
    for (int which = 0; which < 2; ++which) {
        const T *x = which ? k : q;
        const float *dxh = which ? dkh : dqh;
        T *dx = which ? dk : dq;
        // the scans differentiate with respect to the scaled query qs q^
        const float sc = which ? 1.0f : qs;
        float mu = 0.0f;
        for (int d = 0; d < D; ++d) mu += io<T>::ld(x, b + d);
        mu *= 1.0f / D;
        float var = 0.0f;
        for (int d = 0; d < D; ++d) {
            float c = io<T>::ld(x, b + d) - mu;
            var = fmaf(c, c, var);
        }
        float rs = rsqrtf(var * (1.0f / D));
        float m1 = 0.0f, m2 = 0.0f;
        for (int d = 0; d < D; ++d) {
            float xh = (io<T>::ld(x, b + d) - mu) * rs;
            m1 += sc * dxh[b + d];
            m2 = fmaf(sc * dxh[b + d], xh, m2);
        }
        m1 *= 1.0f / D;
        m2 *= 1.0f / D;
        for (int d = 0; d < D; ++d) {
            float xh = (io<T>::ld(x, b + d) - mu) * rs;
            io<T>::st(dx, b + d, (sc * dxh[b + d] - m1 - xh * m2) * rs);
        }
    }
    for (int d = 0; d < D; ++d) io<T>::st(dv, b + d, dva[b + d]);
}

// Column-slice width (including the ones column) that keeps the LDS state
// of a workgroup under 64 KiB (D = 128, p = 2, whose state is 33 KB per
// column, uses most of the 160 KB of LDS instead).
template <int D, bool P2> struct slice_width;
template <> struct slice_width<16, true> { static constexpr int v = 17; };
template <> struct slice_width<32, true> { static constexpr int v = 17; };
template <> struct slice_width<64, true> { static constexpr int v = 5; };
template <> struct slice_width<16, false> { static constexpr int v = 17; };
template <> struct slice_width<32, false> { static constexpr int v = 33; };
template <> struct slice_width<64, false> { static constexpr int v = 65; };
// D = 128, p = 2: two value columns and the ones column per forward slice
// (8385 features x 3 columns = 101 KB of LDS state; 142 KB per workgroup in all)
template <> struct slice_width<128, true> { static constexpr int v = 3; };
template <> struct slice_width<128, false> { static constexpr int v = 65; };

// Segments per head: enough workgroups for ~256 CUs, at most one per chunk.
struct SegPlan {
    int slices, nseg, cps;
    size_t bytes;   // workspace for the segment states (0 with one segment)
};
template <int D, bool P2>
SegPlan seg_plan(int BH, int N)
{
    constexpr int WS = slice_width<D, P2>::v;
    constexpr int W = WS - 1;
    static_assert(W >= 1, "a forward slice holds at least one value column besides the ones column");
    SegPlan sp;
    sp.slices = (D + W - 1) / W;
    const int nch = (N + CH - 1) / CH;
    long long want = 256 / ((long long)BH * sp.slices);
    if (want < 1) want = 1;
    if (want > nch) want = nch;
    if (want > 65535) want = 65535;
    sp.cps = (int)((nch + want - 1) / want);
    sp.nseg = (nch + sp.cps - 1) / sp.cps;
    sp.bytes = sp.nseg > 1 ? (size_t)BH * sp.slices * sp.nseg * feat<D, P2>::P * WS * sizeof(float)
                           : 0;
    return sp;
}

template <int D, bool P2, typename T, bool DROP = false>
static hipError_t fwd_dispatch(const void *q, const void *k, const void *v, void *out, float *g,
                               int BH, int N, int causal, float qs, void *ws, hipStream_t st,
                               Drop dr = Drop{nullptr, 1.0f, nullptr})
{
    constexpr int WS = slice_width<D, P2>::v;
    const SegPlan sp = seg_plan<D, P2>(BH, N);
    dim3 grid(BH, sp.slices, sp.nseg);
    float *sseg = sp.nseg > 1 ? (float *)ws : nullptr;
    if (sseg) {
        hipLaunchKernelGGL((seg_state_kernel<D, P2, WS, T, DROP>), grid, dim3(NT), 0, st,
                           (const T *)k, (const T *)v, sseg, N, sp.cps, dr);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        constexpr int PWS = feat<D, P2>::P * WS;
        const dim3 pgrid((PWS + NT - 1) / NT, BH * sp.slices);
        if (causal)
            hipLaunchKernelGGL((seg_prefix_kernel<PWS, true>), pgrid, dim3(NT), 0, st, sseg,
                               sp.nseg);
        else
            hipLaunchKernelGGL((seg_prefix_kernel<PWS, false>), pgrid, dim3(NT), 0, st, sseg,
                               sp.nseg);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if constexpr (DROP) {
        if (causal) {
            // after the segment states in the workspace, 256-byte aligned
            const size_t off = (sp.bytes + 255) & ~(size_t)255;
            float *wb = (float *)((char *)ws + off);
            const int nch = (N + CH - 1) / CH;
            hipLaunchKernelGGL((drop_wblk_kernel<D, T>),
                               dim3(BH, nch < 65535 ? nch : 65535, (nch + 65534) / 65535),
                               dim3(NT), 0, st, (const T *)q, (const T *)k, wb, N, qs, dr);
            hipError_t e = hipGetLastError();
            if (e != hipSuccess) return e;
            dr.wblk = wb;
        }
    }
    if (causal)
        hipLaunchKernelGGL((fwd_kernel<D, P2, WS, true, T, DROP>), grid, dim3(NT), 0, st,
                           (const T *)q, (const T *)k, (const T *)v, (T *)out, g, N, sp.cps,
                           (const float *)sseg, qs, dr);
    else
        hipLaunchKernelGGL((fwd_kernel<D, P2, WS, false, T, DROP>), grid, dim3(NT), 0, st,
                           (const T *)q, (const T *)k, (const T *)v, (T *)out, g, N, sp.cps,
                           (const float *)sseg, qs, dr);
    return hipGetLastError();
}

// Backward scans: column slices of the D + 1 columns, and segments of chunks
// (states summed in parallel, then prefix- or suffix-summed) when there are too
// few (head, slice) pairs to fill the CUs.
struct BwdPlan {
    int slices, nseg, cps;
    size_t seg_bytes;
};
template <int D, bool P2>
BwdPlan bwd_plan(int BH, int N)
{
    constexpr int WS = slice_width<D, P2>::v;
    BwdPlan bp;
    bp.slices = (D + 1 + WS - 1) / WS;
    const int nch = (N + CH - 1) / CH;
    long long want = 256 / ((long long)BH * bp.slices);
    if (want < 1) want = 1;
    if (want > nch) want = nch;
    if (want > 65535) want = 65535;
    bp.cps = (int)((nch + want - 1) / want);
    bp.nseg = (nch + bp.cps - 1) / bp.cps;
    bp.seg_bytes = bp.nseg > 1 ? (size_t)BH * bp.slices * bp.nseg * feat<D, P2>::P * WS *
                                     sizeof(float)
                               : 0;
    return bp;
}

template <int D, bool P2, bool CAUSAL, typename T, bool DROP = false>
static hipError_t bwd_dispatch2(const void *q, const void *k, const void *v, const void *o,
                                const void *dout, const float *g, void *dq, void *dk, void *dv,
                                int BH, int N, float qs, float *ws, hipStream_t st,
                                Drop dr = Drop{nullptr, 1.0f, nullptr})
{
    constexpr int WS = slice_width<D, P2>::v;
    constexpr int PWS = feat<D, P2>::P * WS;
    const size_t rows = (size_t)BH * N;
    float *cvec = ws;
    float *dqh = cvec + rows;
    float *dkh = dqh + rows * D;
    float *dva = dkh + rows * D;
    const BwdPlan bp = bwd_plan<D, P2>(BH, N);
    float *sseg = bp.nseg > 1 ? dva + rows * D : nullptr;
    if (!grid_fits((long long)((rows + NT - 1) / NT), NT)) return hipErrorInvalidConfiguration;
    const int rb = (int)((rows + NT - 1) / NT);
    hipLaunchKernelGGL((bwd_rowdot_kernel<D, T>), dim3(rb), dim3(NT), 0, st, (const T *)o,
                       (const T *)dout, g, cvec, rows);
    const int nch = (N + CH - 1) / CH;
    hipLaunchKernelGGL((bwd_intra_kernel<D, P2, CAUSAL, T, DROP>),
                       dim3(BH, nch < 65535 ? nch : 65535, (nch + 65534) / 65535), dim3(NT), 0, st, (const T *)q, (const T *)k, (const T *)v,
                       (const T *)dout, g, cvec, dqh, dkh, dva, N, qs, dr);
    const dim3 grid(BH, bp.slices, bp.nseg);
    const dim3 pgrid((PWS + NT - 1) / NT, BH * bp.slices);
    if (sseg) {
        hipLaunchKernelGGL((bwd_seg_state_kernel<D, P2, WS, 0, T, DROP>), grid, dim3(NT), 0, st,
                           (const T *)q, (const T *)k, (const T *)v, (const T *)dout, g, cvec,
                           sseg, N, qs, bp.cps, dr);
        hipLaunchKernelGGL((seg_prefix_kernel<PWS, CAUSAL, false>), pgrid, dim3(NT), 0, st, sseg,
                           bp.nseg);
    }
    hipLaunchKernelGGL((bwd_qscan_kernel<D, P2, WS, CAUSAL, T, DROP>), grid, dim3(NT), 0, st,
                       (const T *)q, (const T *)k, (const T *)v, (const T *)dout, g, cvec, dqh,
                       N, qs, (const float *)sseg, bp.cps, dr);
    if (sseg) {
        // the same buffer, reused in stream order for the k-scan's states
        hipLaunchKernelGGL((bwd_seg_state_kernel<D, P2, WS, 1, T>), grid, dim3(NT), 0, st,
                           (const T *)q, (const T *)k, (const T *)v, (const T *)dout, g, cvec,
                           sseg, N, qs, bp.cps);
        hipLaunchKernelGGL((seg_prefix_kernel<PWS, CAUSAL, true>), pgrid, dim3(NT), 0, st, sseg,
                           bp.nseg);
    }
    hipLaunchKernelGGL((bwd_kscan_kernel<D, P2, WS, CAUSAL, T, DROP>), grid, dim3(NT), 0, st,
                       (const T *)q, (const T *)k, (const T *)v, (const T *)dout, g, cvec, dkh,
                       dva, N, qs, (const float *)sseg, bp.cps, dr);
    hipLaunchKernelGGL((bwd_finish_kernel<D, T>), dim3(rb), dim3(NT), 0, st, (const T *)q,
                       (const T *)k, dqh, dkh, dva, (T *)dq, (T *)dk, (T *)dv, rows, qs);
    return hipGetLastError();
}

template <int D, bool P2, typename T>
static hipError_t bwd_dispatch(const void *q, const void *k, const void *v, const void *o,
                               const void *dout, const float *g, void *dq, void *dk, void *dv,
                               int BH, int N, int causal, float qs, float *ws, hipStream_t st)
{
    if (causal)
        return bwd_dispatch2<D, P2, true, T>(q, k, v, o, dout, g, dq, dk, dv, BH, N, qs, ws, st);
    return bwd_dispatch2<D, P2, false, T>(q, k, v, o, dout, g, dq, dk, dv, BH, N, qs, ws, st);
}

// Keep bits with Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC 2011): one
// thread per mask word (32 features = 8 generator calls).  Feature t of
// token n of head h draws from counter (n, t / 4, h, 0) under the key
// (seed low word, seed high word), output word t % 4, and is kept iff that
// word is >= thr = floor(rate 2^32).
__device__ __forceinline__ void philox4x32_10(uint32_t c[4], uint32_t k0, uint32_t k1)
{
#pragma unroll
    for (int round = 0; round < 10; ++round) {
        const uint32_t hi0 = __umulhi(0xD2511F53u, c[0]), lo0 = 0xD2511F53u * c[0];
        const uint32_t hi1 = __umulhi(0xCD9E8D57u, c[2]), lo1 = 0xCD9E8D57u * c[2];
        const uint32_t n0 = hi1 ^ c[1] ^ k0, n2 = hi0 ^ c[3] ^ k1;
        c[0] = n0;
        c[1] = lo1;
        c[2] = n2;
        c[3] = lo0;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
}

template <int D>
__global__ __launch_bounds__(NT) void dropout_mask_kernel(uint32_t *__restrict__ bits,
                                                          size_t words, int N, uint32_t thr,
                                                          uint32_t key0, uint32_t key1)
{
    constexpr int NW = mask_words(D);
    constexpr int NPAIR = D * (D + 1) / 2;
    const size_t stride = (size_t)gridDim.x * NT;
    for (size_t idx = (size_t)blockIdx.x * NT + threadIdx.x; idx < words; idx += stride) {
        const size_t row = idx / NW;
        const int w = (int)(idx % NW);
        const uint32_t n = (uint32_t)(row % (size_t)N), head = (uint32_t)(row / (size_t)N);
        uint32_t word = 0;
#pragma unroll
        for (int g4 = 0; g4 < 8; ++g4) {
            const int t0 = 32 * w + 4 * g4;
            if (t0 >= NPAIR) break;
            uint32_t c[4] = {n, (uint32_t)(t0 >> 2), head, 0u};
            philox4x32_10(c, key0, key1);
#pragma unroll
            for (int u = 0; u < 4; ++u)
                if (t0 + u < NPAIR && c[u] >= thr) word |= 1u << (4 * g4 + u);
        }
        bits[idx] = word;
    }
}

}  // namespace generic

hipError_t dropout_mask(uint32_t *bits, int BH, int N, int D, uint32_t thr, uint64_t seed,
                        hipStream_t st)
{
    using namespace generic;
    const size_t words = (size_t)BH * N * (size_t)mask_words(D);
    // grid-stride: at most 2^20 workgroups (enough to fill the chip many times)
    const size_t want = (words + NT - 1) / NT;
    const dim3 grid((unsigned)(want < ((size_t)1 << 20) ? want : ((size_t)1 << 20)));
    const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
    switch (D) {
    case 16: hipLaunchKernelGGL((dropout_mask_kernel<16>), grid, dim3(NT), 0, st, bits, words, N, thr, k0, k1); break;
    case 32: hipLaunchKernelGGL((dropout_mask_kernel<32>), grid, dim3(NT), 0, st, bits, words, N, thr, k0, k1); break;
    case 64: hipLaunchKernelGGL((dropout_mask_kernel<64>), grid, dim3(NT), 0, st, bits, words, N, thr, k0, k1); break;
    default: hipLaunchKernelGGL((dropout_mask_kernel<128>), grid, dim3(NT), 0, st, bits, words, N, thr, k0, k1); break;
    }
    return hipGetLastError();
}

template <typename T>
static hipError_t drop_fwd_t(const void *q, const void *k, const void *v, void *out, float *g,
                             int BH, int N, int D, int causal, float qs, const uint32_t *bits,
                             float inv, void *ws, hipStream_t st)
{
    using namespace generic;
    const Drop dr{bits, inv, nullptr};
    switch (D) {
    case 16: return fwd_dispatch<16, true, T, true>(q, k, v, out, g, BH, N, causal, qs, ws, st, dr);
    case 32: return fwd_dispatch<32, true, T, true>(q, k, v, out, g, BH, N, causal, qs, ws, st, dr);
    case 64: return fwd_dispatch<64, true, T, true>(q, k, v, out, g, BH, N, causal, qs, ws, st, dr);
    default: return fwd_dispatch<128, true, T, true>(q, k, v, out, g, BH, N, causal, qs, ws, st, dr);
    }
}

template <int D, typename T>
static hipError_t drop_bwd_d(const void *q, const void *k, const void *v, const void *o,
                             const void *dout, const float *g, void *dq, void *dk, void *dv,
                             int BH, int N, int causal, float qs, float *ws, hipStream_t st,
                             generic::Drop dr)
{
    using namespace generic;
    if (causal)
        return bwd_dispatch2<D, true, true, T, true>(q, k, v, o, dout, g, dq, dk, dv, BH, N, qs,
                                                     ws, st, dr);
    return bwd_dispatch2<D, true, false, T, true>(q, k, v, o, dout, g, dq, dk, dv, BH, N, qs, ws,
                                                  st, dr);
}

template <typename T>
static hipError_t drop_bwd_t(const void *q, const void *k, const void *v, const void *o,
                             const void *dout, const float *g, void *dq, void *dk, void *dv,
                             int BH, int N, int D, int causal, float qs, const uint32_t *bits,
                             float inv, float *ws, hipStream_t st)
{
    const generic::Drop dr{bits, inv, nullptr};
    switch (D) {
    case 16: return drop_bwd_d<16, T>(q, k, v, o, dout, g, dq, dk, dv, BH, N, causal, qs, ws, st, dr);
    case 32: return drop_bwd_d<32, T>(q, k, v, o, dout, g, dq, dk, dv, BH, N, causal, qs, ws, st, dr);
    case 64: return drop_bwd_d<64, T>(q, k, v, o, dout, g, dq, dk, dv, BH, N, causal, qs, ws, st, dr);
    default: return drop_bwd_d<128, T>(q, k, v, o, dout, g, dq, dk, dv, BH, N, causal, qs, ws, st, dr);
    }
}

size_t generic_fwd_dropout_workspace(int BH, int N, int D, int causal)
{
    const size_t seg = generic_fwd_workspace(BH, N, D, 2);
    if (!causal) return seg;
    const size_t nch = ((size_t)N + generic::CH - 1) / generic::CH;
    return ((seg + 255) & ~(size_t)255) +
           (size_t)BH * nch * generic::CH * generic::CH * sizeof(float);
}

hipError_t generic_fwd_dropout(const void *q, const void *k, const void *v, void *out, float *g,
                               int BH, int N, int D, int causal, int is_bf16, float qs,
                               const uint32_t *bits, float inv, void *ws, hipStream_t st)
{
    if (is_bf16) return drop_fwd_t<bf16_t>(q, k, v, out, g, BH, N, D, causal, qs, bits, inv, ws, st);
    return drop_fwd_t<float>(q, k, v, out, g, BH, N, D, causal, qs, bits, inv, ws, st);
}

hipError_t generic_bwd_dropout(const void *q, const void *k, const void *v, const void *o,
                               const void *dout, const float *g, void *dq, void *dk, void *dv,
                               int BH, int N, int D, int causal, int is_bf16, float qs,
                               const uint32_t *bits, float inv, void *ws, hipStream_t st)
{
    if (is_bf16)
        return drop_bwd_t<bf16_t>(q, k, v, o, dout, g, dq, dk, dv, BH, N, D, causal, qs, bits,
                                  inv, (float *)ws, st);
    return drop_bwd_t<float>(q, k, v, o, dout, g, dq, dk, dv, BH, N, D, causal, qs, bits, inv,
                             (float *)ws, st);
}

size_t generic_bwd_workspace(int B, int H, int N, int D, int p)
{
    using namespace generic;
    const size_t rows = (size_t)B * H * N;
    const int BH = B * H;
    size_t seg = 0;
    if (D == 16) seg = p == 2 ? bwd_plan<16, true>(BH, N).seg_bytes : bwd_plan<16, false>(BH, N).seg_bytes;
    else if (D == 32) seg = p == 2 ? bwd_plan<32, true>(BH, N).seg_bytes : bwd_plan<32, false>(BH, N).seg_bytes;
    else if (D == 64) seg = p == 2 ? bwd_plan<64, true>(BH, N).seg_bytes : bwd_plan<64, false>(BH, N).seg_bytes;
    else seg = p == 2 ? bwd_plan<128, true>(BH, N).seg_bytes : bwd_plan<128, false>(BH, N).seg_bytes;
    return sizeof(float) * (rows + 3 * rows * (size_t)D) + seg;
}

#define FM_DISPATCH_D_P(FN, D, p, ...)                                   \
    ((D) == 16 ? ((p) == 2 ? FN<16, true, T>(__VA_ARGS__) : FN<16, false, T>(__VA_ARGS__)) : \
     (D) == 32 ? ((p) == 2 ? FN<32, true, T>(__VA_ARGS__) : FN<32, false, T>(__VA_ARGS__)) : \
     (D) == 64 ? ((p) == 2 ? FN<64, true, T>(__VA_ARGS__) : FN<64, false, T>(__VA_ARGS__)) : \
                 ((p) == 2 ? FN<128, true, T>(__VA_ARGS__) : FN<128, false, T>(__VA_ARGS__)))

template <typename T>
static hipError_t gen_fwd_t(const void *q, const void *k, const void *v, void *out, float *g,
                            int BH, int N, int D, int p, int causal, float qs, void *ws,
                            hipStream_t st)
{
    return FM_DISPATCH_D_P(generic::fwd_dispatch, D, p, q, k, v, out, g, BH, N, causal, qs, ws,
                           st);
}

size_t generic_fwd_workspace(int BH, int N, int D, int p)
{
    using namespace generic;
    if (D == 16) return p == 2 ? seg_plan<16, true>(BH, N).bytes : seg_plan<16, false>(BH, N).bytes;
    if (D == 32) return p == 2 ? seg_plan<32, true>(BH, N).bytes : seg_plan<32, false>(BH, N).bytes;
    if (D == 64) return p == 2 ? seg_plan<64, true>(BH, N).bytes : seg_plan<64, false>(BH, N).bytes;
    return p == 2 ? seg_plan<128, true>(BH, N).bytes : seg_plan<128, false>(BH, N).bytes;
}

template <typename T>
static hipError_t gen_bwd_t(const void *q, const void *k, const void *v, const void *o,
                            const void *dout, const float *g, void *dq, void *dk, void *dv,
                            int BH, int N, int D, int p, int causal, float qs, float *ws,
                            hipStream_t st)
{
    return FM_DISPATCH_D_P(generic::bwd_dispatch, D, p, q, k, v, o, dout, g, dq, dk, dv, BH, N,
                           causal, qs, ws, st);
}

hipError_t generic_fwd(const void *q, const void *k, const void *v, void *out, float *g, int BH,
                       int N, int D, int p, int causal, int is_bf16, float qs, void *ws,
                       hipStream_t st)
{
    if (is_bf16) return gen_fwd_t<bf16_t>(q, k, v, out, g, BH, N, D, p, causal, qs, ws, st);
    return gen_fwd_t<float>(q, k, v, out, g, BH, N, D, p, causal, qs, ws, st);
}

hipError_t generic_bwd(const void *q, const void *k, const void *v, const void *o,
                       const void *dout, const float *g, void *dq, void *dk, void *dv, int BH,
                       int N, int D, int p, int causal, int is_bf16, float qs, void *ws,
                       hipStream_t st)
{
    if (is_bf16)
        return gen_bwd_t<bf16_t>(q, k, v, o, dout, g, dq, dk, dv, BH, N, D, p, causal, qs,
                                 (float *)ws, st);
    return gen_bwd_t<float>(q, k, v, o, dout, g, dq, dk, dv, BH, N, D, p, causal, qs,
                            (float *)ws, st);
}

}  // namespace fm

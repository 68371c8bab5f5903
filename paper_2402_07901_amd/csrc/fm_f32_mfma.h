// Shared pieces of the float32 MFMA kernels (v_mfma_f32_16x16x4_f32, p = 2):
// the forward and backward scans of fm_f32_mfma.hip and fm_f32_bwd.hip.
//
// MFMA lane layout (16x16x4 f32, lane = 16h + r16): A holds row r16, K index
// h; B holds column r16, K index h; the accumulator holds column r16, rows
// 4h..4h+3.  Contractions over 16 rows of an accumulator run as four K steps
// i = 0..3 with K index h <-> row 4h + i, so element i of an accumulator is
// directly the A operand of step i (no data movement).
//
// Feature tiles (16 features of phi(k) = [k_l, (k_m k_l)] x 16 value
// columns): the linear tiles u (features k_l, l = 16u..16u+15) and the
// quadratic tiles (m, u) for u >= m/16 (features k_m k_l); a diagonal tile
// u = m/16 holds both (m, l) and (l, m) of its block.  Wave gw (over the
// parts of a head and slice) owns the linear tile u = gw (gw < D/16) and the
// quadratic tiles of its channels chan(c, class, gw), c < D / (waves * parts).
#pragma once

#include <hip/hip_runtime.h>

#include <stddef.h>

#include <type_traits>

#include "fm_common.h"
#include "fm_mfma.h"

namespace fm {
namespace m32 {

using mx::static_for;
typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int C = 32;      // tokens per chunk
constexpr int SL = 16;     // value columns per workgroup
constexpr int TARGET_BLOCKS = 256;

__device__ __forceinline__ f4 mma(float a, float b, f4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// P: the order of the Taylor weight (1: f = 1 + s, state = the linear tiles
// only; 2: f = 1 + s + s^2/2, plus the quadratic tiles and Y3).
template <int D, int P = 2>
struct Pat {
    // Workgroups sharing one (head, slice) and waves per workgroup.  D = 128,
    // p = 2 has too many feature tiles for one workgroup's accumulators: four
    // workgroups each take a quarter of them (and a quarter of the Y3 rows)
    // and write partial F, G.  Eight waves (two per SIMD) keep at most about
    // 84 state registers each, so a second wave hides each wave's stalls.
    static constexpr int NPART = (P == 2 && D == 128) ? 4 : 1;
    static constexpr int NW = 8;
    static constexpr int NTH = NW * 64;
    static constexpr int LPT = NTH / C;                // staging lanes per token
    static constexpr int DP = D / LPT;                 // staged channels per lane
    static constexpr int VPL = SL / LPT;               // staged value columns per lane
    static constexpr int NU = D / 16;                  // 16-channel blocks
    static constexpr int NGW = NW * NPART;             // waves over the parts
    static constexpr int NCH = D / NGW;                // channels per wave
    // Block u0 of the wave's c-th channel.  Up to 16 waves: channel
    // m = gw + NGW c, in block NGW c / 16.  With 32 waves (two wave classes
    // gh = gw / 16, one per pair of workgroups) wave gw takes channel
    // 16 u0 + gw % 16 of block u0 = 2c + ((c & 1) ^ gh): blocks 0, 3, 4, 7
    // for class 0 and 1, 2, 5, 6 for class 1, so that both classes hold the
    // same number of tiles (sum over c of NU - u0); the plain order 2c + gh
    // would give class 0 NCH more tiles than class 1, and the workgroups of
    // that class would set the pace.
    static constexpr int NH = NGW > 16 ? NGW / 16 : 1;  // wave classes
    static constexpr int u0(int c, int gh) { return NGW > 16 ? 2 * c + ((c & 1) ^ gh) : NGW * c / 16; }
    __device__ static int chan(int c, int gh, int gw) { return NGW > 16 ? 16 * u0(c, gh) + (gw & 15) : gw + NGW * c; }
    // first tile of channel c (its diagonal tile; u runs from u0 to NU-1)
    static constexpr int first(int c, int gh)
    {
        int t = 1;
        for (int cc = 0; cc < c; ++cc) t += NU - u0(cc, gh);
        return t;
    }
    // quadratic tiles per wave (the larger class)
    static constexpr int NQ = P != 2 ? 0 : first(NCH, 0) > first(NCH, NH - 1) ? first(NCH, 0) - 1 : first(NCH, NH - 1) - 1;
    static constexpr int NT = 1 + NQ;                  // + the linear slot
    static constexpr int NLB = NU / NPART;             // Y3 row blocks per part
    // the denominator's contraction over each Y3 row block: split over KQ
    // waves by K range where one workgroup holds two blocks of 128 channels
    // (every wave takes a share), else on the last NLB waves whole
    static constexpr int KQ = (P == 2 && NPART > 1) ? NW / NLB : 1;
    static constexpr int NGI = NLB * KQ;               // partial sums per token
    static constexpr int Y3R = P == 2 ? 16 * NLB : 0;  // Y3 rows per part
    // Y3 tiles per part: one part keeps the blocks u <= u2 and mirrors them,
    // several parts keep full rows
    static constexpr int NY3 = P != 2 ? 0 : NPART == 1 ? NU * (NU + 1) / 2 : NLB * NU;
    static constexpr int RS = D + 2;   // row stride of row-major tiles (floats)
    static constexpr int TS = C + 2;   // row stride of transposed tiles
    static_assert(NGW <= 16 ? 16 % NGW == 0 : NGW == 32 && NCH % 2 == 0, "channel blocks");
    static_assert(LPT * C == NTH && DP * LPT == D && VPL * LPT == SL, "staging");
};

// Runs f(integral_constant<int, gh>) for the workgroup's wave class gh.
template <int D, int P, typename F>
__device__ __forceinline__ void with_wave_class(int gw, F &&f)
{
    if constexpr (Pat<D, P>::NH == 1) {
        f(std::integral_constant<int, 0>{});
    } else {
        if (gw < 16) f(std::integral_constant<int, 0>{});
        else f(std::integral_constant<int, 1>{});
    }
}

enum Mode { DELTA = 0, SCAN = 1, QUERY = 2, BOTH = 3 };

// NE consecutive elements of T (bf16 or float) as raw 32-bit words, loaded as
// one access of their size (the rows are 16-byte aligned and NE * sizeof(T)
// divides the row) and converted to float only where they are used: a
// prefetch into these registers does not wait for its loads.
template <typename T, int NE>
struct RawRow {
    static constexpr int BYTES = NE * (int)sizeof(T);
    static constexpr int NWD = BYTES < 4 ? 1 : BYTES / 4;
    static_assert(BYTES == 2 || BYTES == 4 || BYTES == 8 || BYTES % 16 == 0, "row piece");
    uint32_t w[NWD];
    __device__ __forceinline__ void load(const T *p, bool valid)
    {
        if constexpr (BYTES == 2) {
            w[0] = 0u;
            if (valid) w[0] = *(const uint16_t *)p;
        } else if constexpr (BYTES == 4) {
            w[0] = 0u;
            if (valid) w[0] = *(const uint32_t *)p;
        } else if constexpr (BYTES == 8) {
            uint2 x = make_uint2(0u, 0u);
            if (valid) x = *(const uint2 *)p;
            w[0] = x.x;
            w[1] = x.y;
        } else {
#pragma unroll
            for (int j = 0; j < BYTES / 16; ++j) {
                uint4 x = make_uint4(0u, 0u, 0u, 0u);
                if (valid) x = ((const uint4 *)p)[j];
                w[4 * j] = x.x;
                w[4 * j + 1] = x.y;
                w[4 * j + 2] = x.z;
                w[4 * j + 3] = x.w;
            }
        }
    }
    // element i (a compile-time index after unrolling)
    __device__ __forceinline__ float get(int i) const
    {
        if constexpr (sizeof(T) == 4) return __uint_as_float(w[i]);
        else return __uint_as_float((i & 1) ? (w[i >> 1] & 0xffff0000u) : (w[i >> 1] << 16));
    }
};

// Sum over an aligned row of 16 lanes, in every lane, with DPP moves (no LDS
// round trip): swap neighbours, swap pairs, mirror the quads of each half
// row, mirror the half rows.
__device__ __forceinline__ float row16_sum(float x)
{
    x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0xB1, 0xF, 0xF, true));
    x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x4E, 0xF, 0xF, true));
    x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x141, 0xF, 0xF, true));
    x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x140, 0xF, 0xF, true));
    return x;
}

// Standardises the channels this thread holds of its token (Sec. 2.2, Eqs.
// 6-7: population std, no epsilon; the token's LPT = 16 lanes form one DPP
// row) and scales them.  Every lane of the wave must take part.
template <int D>
__device__ __forceinline__ void standardise_part(float (&x)[Pat<D>::DP], bool valid, float scale)
{
    constexpr int DP = Pat<D>::DP;
    static_assert(Pat<D>::LPT == 16, "one DPP row per token");
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < DP; ++i) s += x[i];
    s = row16_sum(s);
    const float mu = s * (1.0f / D);
    float v = 0.f;
#pragma unroll
    for (int i = 0; i < DP; ++i) {
        x[i] -= mu;
        v = fmaf(x[i], x[i], v);
    }
    v = row16_sum(v);
    const float r = valid ? __builtin_amdgcn_rsqf(v * (1.0f / D)) * scale : 0.0f;
#pragma unroll
    for (int i = 0; i < DP; ++i) x[i] *= r;
}

// In-chunk block (row tile rt, key tile st <= rt) of a 32-token chunk: the
// part that adds it to its partial F and G.
template <int NPART>
__host__ __device__ constexpr int inchunk_owner(int rt, int st)
{
    return (rt * (rt + 1) / 2 + st) % NPART;
}

// Segment sums -> exclusive prefix over segments (causal) or the total in
// every segment (non-causal), in place; one thread per float of one item.
static __global__ __launch_bounds__(256) void prefix_kernel(float *__restrict__ sums, int nseg,
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

inline int nseg_of(int items, int nch, int target = TARGET_BLOCKS)
{
    int s = target / (items > 0 ? items : 1);
    if (s < 1) s = 1;
    if (s > nch) s = nch;
    return s;
}

inline size_t a256(size_t b) { return (b + 255) & ~(size_t)255; }

}  // namespace m32
}  // namespace fm

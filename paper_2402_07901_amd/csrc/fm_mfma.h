// Device helpers shared by the D = 64, p = 2 MFMA kernels (causal scan,
// non-causal moment build and query contraction, backward): fp16 operand packing for
// v_mfma_f32_16x16x32_f16, the per-wave feature-tile pattern of the moment
// state, LDS row padding and per-token standardisation (Sec. 2.2, Eqs. 6-7).
//
// MFMA 16x16x32 lane layout (lane = 16h + r16): the A operand holds row r16,
// K indices 8h..8h+7; the B operand holds column r16, the same K indices; the
// accumulator holds column r16, rows 4h..4h+3.
//
// Feature tiles.  The quadratic features k_m k_l are grouped in 16x16 tiles
// (m, u): rows l = 16u..16u+15 for one m, with u >= m/16 (symmetric tiles:
// 160 of them) plus 4 linear tiles (k_l) -- 2624 feature rows instead of the
// 4160 of the full square, 2080 + 65 being the minimum.  A "diagonal" tile
// (u == m/16) carries both (m,l) and (l,m) and enters the query contraction
// with weight 1/2, the others with weight 1, so psi(q).phi(k) = 1 + s + s^2/2
// exactly (constant term separate).  The eight-wave pattern below (wave w
// owns the tiles of m = w (mod 8) and, for w < 4, the linear tile u = w: 21
// tiles) serves the non-causal moment build; the causal scan defines its own
// four-wave pattern of 41 tiles.
//
// Pairing for the query contraction: K step p combines tiles 2p and 2p+1;
// K index 8h+r <-> tile 2p row 4h+r, 8h+4+r <-> tile 2p+1 row 4h+r, which is
// exactly the accumulator layout of the two tiles, so a state accumulator
// converted to fp16 is directly an A operand.
#pragma once

#include <hip/hip_runtime.h>

#include <stdint.h>

#include <type_traits>

#include "fm_common.h"

namespace fm {
namespace mx {

typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef _Float16 h4 __attribute__((ext_vector_type(4)));
typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int D = 64;

template <int I, int N, typename F>
__device__ __forceinline__ void static_for(F &&f)
{
    if constexpr (I < N) {
        f(std::integral_constant<int, I>{});
        static_for<I + 1, N>(f);
    }
}

// Tiles of a wave w: tile 0 is the linear tile u = w (waves 0..3 only; it
// stays zero in waves 4..7), then for the wave's channels m = w + 8*idx
// (idx = 0..7) the tiles u = idx/2 .. 3 (m/16 == idx/2 for every w < 8), so
// all waves share one tile pattern: 1 + 4+4+3+3+2+2+1+1 = 21 tiles.
constexpr int NT = 21;
constexpr int NKS = (NT + 1) / 2;   // K steps of the query contraction
__host__ __device__ constexpr int u0_of(int idx) { return idx / 2; }
__host__ __device__ constexpr int first_tile(int idx)
{
    int t = 1;
    for (int i = 0; i < idx; ++i) t += 4 - u0_of(i);
    return t;
}
struct Tile {
    int kind;  // 0 linear, 1 quadratic, -1 padding
    int idx;   // channel m = w + 8*idx
    int u;     // l tile
};
__host__ __device__ constexpr Tile tile_of(int t)
{
    if (t == 0) return Tile{0, -1, -1};
    for (int idx = 0; idx < 8; ++idx)
        if (t < first_tile(idx) + 4 - u0_of(idx)) return Tile{1, idx, u0_of(idx) + t - first_tile(idx)};
    return Tile{-1, -1, -1};
}
__host__ __device__ constexpr bool is_diag(int t)
{
    return t < NT && tile_of(t).kind == 1 && tile_of(t).u == u0_of(tile_of(t).idx);
}

// Y3 tiles (u <= u2), 10 of them: waves 0 and 1 own two, the others one.
__device__ __forceinline__ int y3_count(int w) { return w < 2 ? 2 : 1; }
__device__ __forceinline__ void y3_tile(int w, int k, int &u, int &u2)
{
    // tile i of the upper triangle in row order (0,0) (0,1) .. (3,3), computed
    // rather than looked up in a table (which would live in global memory)
    const int i = w < 2 ? 2 * w + k : 2 + w;
    u = (i >= 4) + (i >= 7) + (i >= 9);
    u2 = i - (4 * u - (u * (u - 1)) / 2) + u;
}

// LDS rows are padded by 16 bytes: 16 lanes reading the same column of 16
// consecutive rows then fall on 16 distinct 4-bank groups, and offsets stay
// affine so constant parts fold into the instructions.  Offsets in halves.
constexpr int RS64 = 64 + 8;     // rows of 64 halves
constexpr int RS128 = 128 + 8;   // rows of 128 halves
__device__ __forceinline__ int sw64(int row, int col) { return row * RS64 + col; }
__device__ __forceinline__ int sw128(int row, int col) { return row * RS128 + col; }
// Transposed operands ([channel][token]) staged by lanes that each hold 8
// channels of a few tokens write rows 8 apart in one store instruction, which
// the padding maps to the same banks.  XOR-ing the column (in 16-byte units)
// with the row's group of 8 spreads those stores over all banks and keeps
// every aligned 8- or 16-byte read contiguous.  Used where the staging
// stores dominate (the backward's scans); the forward kernels keep plain
// padding, whose reads need no per-lane address work.
__device__ __forceinline__ int swx(int row, int col) { return row * RS128 + (col ^ (((row >> 3) & 7) << 3)); }


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

// Sum over an aligned octet of lanes with DPP: swap neighbours, swap pairs,
// then mirror the two quads of each half row.
__device__ __forceinline__ float octet_sum(float x)
{
    x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0xB1, 0xF, 0xF, true));
    x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x4E, 0xF, 0xF, true));
    x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x141, 0xF, 0xF, true));
    return x;
}

// Standardises the 8 channels this lane holds of one token (the token's 64
// channels are spread over the 8 lanes of an aligned octet) and returns them
// as fp16.  Population variance, no epsilon; invalid rows become zero.
// `scale` multiplies the standardised row (the score scale of the query side;
// 1 leaves it unchanged).
__device__ __forceinline__ h8 standardise8(const float *xin, bool valid, float scale = 1.0f)
{
    float x[8];
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) s += xin[i];
    const float mu = octet_sum(s) * (1.0f / D);
    float v = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        x[i] = xin[i] - mu;
        v = fmaf(x[i], x[i], v);
    }
    const float r = valid ? __builtin_amdgcn_rsqf(octet_sum(v) * (1.0f / D)) * scale : 0.0f;
    h8 o;
#pragma unroll
    for (int i = 0; i < 8; i += 2) {
        const h2 pr = {(_Float16)(x[i] * r), (_Float16)(x[i + 1] * r)};
        o[i] = pr[0];
        o[i + 1] = pr[1];
    }
    return o;
}

// Two floats -> two bf16 (round to nearest even, v_cvt_pk_bf16_f32) packed
// low-first into one word.
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b)
{
    typedef __bf16 bf2 __attribute__((ext_vector_type(2)));
    typedef float fl2 __attribute__((ext_vector_type(2)));
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(fl2{a, b}, bf2));
}

// sum of 8 halves in fp32 (dot products with ones)
__device__ __forceinline__ float hsum8(h8 a)
{
    const h2 one = {(_Float16)1.0f, (_Float16)1.0f};
    float s = 0.f;
    s = __builtin_amdgcn_fdot2(h2{a[0], a[1]}, one, s, false);
    s = __builtin_amdgcn_fdot2(h2{a[2], a[3]}, one, s, false);
    s = __builtin_amdgcn_fdot2(h2{a[4], a[5]}, one, s, false);
    s = __builtin_amdgcn_fdot2(h2{a[6], a[7]}, one, s, false);
    return s;
}

}  // namespace mx
}  // namespace fm

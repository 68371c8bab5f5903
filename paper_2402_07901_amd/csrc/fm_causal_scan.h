// The causal MFMA scan (D = 64, p = 2) as a device function, shared by the
// forward launch (csrc/fm_causal_mfma.hip) and the backward's combined
// dv / moment-gradient launch (csrc/fm_bwd_mfma.hip).
//
// Chunked causal scan (Sec. 2.4, causal moments "xcausal"/"ycausal" carried
// across chunks of 128 tokens instead of per row).  One workgroup owns one
// (batch, head, slice of 16 value columns) and keeps the moment state
// S[f][j] = sum_n phi_f(k^_n) v_nj of the slice on chip for the whole
// sequence; the state never touches HBM.
//
// Two kinds of waves share each SIMD:
//  * state waves 0..3 hold the state as fp16 MFMA operands (41 feature tiles
//    of 16 rows each, 84 registers per lane) and do the two contractions
//    against it: the query contraction F^T += S^T Psi(Q)^T (Psi generated in
//    registers with packed fp16 multiplies) and the state update
//    S += Phi(K)^T V;
//  * helper waves 4..7 stage the next chunk (q^ and k^, standardised once per
//    call by standardise_qk (Sec. 2.2, Eqs. 6-7) and read in fp16; transposes;
//    scaled v), compute the in-chunk block tril(f(Q K^T)) V on MFMA and
//    the denominators G_i = n0 + q.y2 + 1/2 q^T Y3 q + in-chunk row sums,
//    and combine the partial numerators into O = F / G.
// Per chunk there are two phases separated by barriers: (1) query
// contraction | in-chunk block and denominators; (2) state update | output,
// prefix sums, Y3 update and staging of the next chunk.  The two kinds of
// work overlap on each SIMD instead of running in lockstep.
//
// Segments (load balance, Sec. 2.4's causal recurrences cut at a chunk
// boundary).  When a launch of one workgroup per (head, slice) would leave
// the GPU's CUs idle for part of the time (e.g. 384 workgroups on 256 CUs),
// each (head, slice) is scanned by two workgroups: segment 0 takes the
// chunks before csplit and, at its end, writes its summary -- the moment
// state, Y3, y2 and x1 accumulated over those chunks, i.e. the exclusive
// prefix of segment 1 -- and raises a flag; segment 1 waits for the flag
// (bounded), loads the summary and scans the remaining chunks from it.  The
// second segments come after all first segments in the grid, so they are
// dispatched after them.  If the flag does not come within the bound, the
// segment builds the prefix itself (state updates and prefix sums over the
// earlier chunks, no outputs), so the result never depends on the order in
// which workgroups run.  Both segments scale v from the whole slice's max|v|
// and perform the same operations in the same order as one workgroup over
// all chunks: split and unsplit scans give bit-identical results.
//
// State numerics.  The state lives in fp16 (v is pre-scaled by a power of two
// 2^-e per workgroup so that no entry, bounded by N * 63 * max|v|, can exceed
// 2^15).  A tile's accumulator layout holds exactly the elements of its half of
// the paired operand, so each update accumulates the chunk's contribution in
// fp32 from zero, rounds it to fp16 and adds it to the state with packed fp16
// arithmetic (two roundings per chunk).  Diagonal tiles are stored halved (the
// 1/2 of f_2) and take half the contribution.
#pragma once

#include <hip/hip_runtime.h>

#include <type_traits>

#include "fm_common.h"
#include "fm_mfma.h"

namespace fm {
namespace mfma_causal {

using namespace mx;

constexpr int C = 128;        // tokens per chunk
constexpr int NRT = C / 16;   // 16-token row tiles per chunk
constexpr int NKS2 = C / 32;  // 32-token K steps of the state update
constexpr int NSW = 4;        // state waves (one per SIMD)
constexpr int NW = 8;         // waves per workgroup
constexpr int NTH = NW * 64;
constexpr int NHT = NTH - NSW * 64;  // helper threads
constexpr int SL = 16;        // value columns per workgroup
constexpr int NSL = D / SL;

// Feature tiles of state wave w: tile 0 is the linear tile u = w (features
// k_l, l = 16w..16w+15); then for the wave's channels
// m = 16 (i/4) + 4w + i%4 (i = 0..15: channels 4w..4w+3 of each 16-channel
// block, so a lane reads them as four 4-channel groups of a row-major q^ row)
// the quadratic tiles (m, u) for u = i/4 .. 3 (m/16 == i/4):
// 1 + 4*(4+3+2+1) = 41 tiles; 164 over the four waves.
constexpr int NQ = 16;
__host__ __device__ constexpr int u0_of(int i) { return i / 4; }
__host__ __device__ constexpr int first_tile(int i)
{
    int t = 1;
    for (int j = 0; j < i; ++j) t += 4 - u0_of(j);
    return t;
}
constexpr int NT = first_tile(NQ);    // 41
constexpr int NKS = (NT + 1) / 2;     // 21 K steps of the query contraction
struct Tile {
    int kind;  // 0 linear, 1 quadratic, -1 padding
    int i;     // channel m = 16 (i/4) + 4w + i%4
    int u;     // l tile
};
__host__ __device__ constexpr Tile tile_of(int t)
{
    if (t == 0) return Tile{0, -1, -1};
    for (int i = 0; i < NQ; ++i)
        if (t < first_tile(i) + 4 - u0_of(i)) return Tile{1, i, u0_of(i) + t - first_tile(i)};
    return Tile{-1, -1, -1};
}
static_assert(NT == 41 && tile_of(40).kind == 1 && tile_of(41).kind == -1, "tile pattern");
// The first tile of each channel (u = i/4) is its diagonal tile.
static_assert(tile_of(first_tile(5)).u == u0_of(5) && tile_of(first_tile(5)).i == 5, "tile pattern");

// Y3 tiles (u <= u2), 10 of them: helpers 0 and 1 own three, 2 and 3 two.
__device__ __forceinline__ int y3_count(int hw) { return hw < 2 ? 3 : 2; }
// Tile i of the upper triangle in row order: (0,0) (0,1) (0,2) (0,3) (1,1)
// ... (3,3); computed, not looked up (a table would be placed in memory and
// each lookup would wait on a global load).
__device__ __forceinline__ void y3_tile(int hw, int kk, int &u, int &u2)
{
    const int i = hw < 2 ? 3 * hw + kk : 6 + 2 * (hw - 2) + kk;
    u = (i >= 4) + (i >= 7) + (i >= 9);
    u2 = i - (4 * u - (u * (u - 1)) / 2) + u;
}

struct Smem {
    _Float16 qrow[C * RS64];        // q^ [token][m]
    _Float16 krow[C * RS64];        // k^ [token][m]
    _Float16 kT[2][D * RS128];      // k^ [m][token], double-buffered by chunk parity
    _Float16 vT[2][SL * RS128];     // scaled v [j][token], double-buffered
    _Float16 y3h[D * RS64];         // scaled Y3 (prefix before the chunk)
    float fpart[NSW * C * SL];      // partial F^T of the state waves: [wave][column quad][token][4]
    alignas(16) float y2[2][D];     // sum k^ before the chunk (by chunk parity)
    alignas(16) float y2s[2][D];    // the same times 2^(1-gexp), gexp the Y3 scale
    alignas(16) float x1[2][SL];    // sum of scaled v before the chunk
    float red[NW];
    int segok;                      // the summary of segment 0 arrived
};

// Two-segment split of a scan (see "Segments" above).
struct SegArgs {
    unsigned char *sum;     // summaries, SUM_BYTES per (head, slice); null if no split
    unsigned int *flags;    // one per (head, slice), zeroed before the launch
    int split;              // 0: one workgroup per (head, slice); 1: two
    int csplit;             // first chunk of segment 1
    int wait;               // 1: segment 1 waits for segment 0's summary; 0: rebuilds it
};
// summary layout: fp16 state [wave][pair][lane] (h8), Y3 accumulators
// [helper][tile][lane] (f4), y2, y2 scaled, x1 (fp32)
constexpr size_t SUM_AST = (size_t)NSW * NKS * 64 * 16;
constexpr size_t SUM_Y3 = (size_t)4 * 3 * 64 * 16;
constexpr size_t SUM_MISC = (size_t)(D + D + SL) * 4;
constexpr size_t SUM_BYTES = (SUM_AST + SUM_Y3 + SUM_MISC + 255) & ~(size_t)255;
// polls of a waiting segment (about 0.3 s at 2 GHz) before it rebuilds the
// prefix itself
constexpr int SEG_SPIN = 1 << 20;

// Summary words are written and read as relaxed atomics at device scope:
// such accesses go to the level where every XCD's CUs see the same data (the
// per-XCD L2s are not coherent with each other), so the flag protocol needs
// no cache-wide write-back or invalidation (which, done by every first
// segment and every second one, cost more than the split gains).  Ordering:
// each thread's summary stores have completed before the workgroup barrier
// that precedes the flag store, and the summary loads are issued after the
// flag load has returned.  A 16-byte per-lane value of a wave is stored
// word-major (8-byte word i of lane l at grp[64 i + l]) so that each store
// writes 512 contiguous bytes: these stores go through to memory, where
// lane-interleaved partial lines cost several times more.
typedef unsigned long long u64x2 __attribute__((ext_vector_type(2)));
template <typename T>
__device__ __forceinline__ void sum_put_lane(unsigned long long *grp, int lane, const T &x)
{
    static_assert(sizeof(T) == 16, "16-byte lane values");
    const u64x2 w = __builtin_bit_cast(u64x2, x);
    __hip_atomic_store(grp + lane, w[0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(grp + 64 + lane, w[1], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <typename T>
__device__ __forceinline__ T sum_get_lane(const unsigned long long *grp, int lane)
{
    static_assert(sizeof(T) == 16, "16-byte lane values");
    u64x2 w;
    w[0] = __hip_atomic_load(grp + lane, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    w[1] = __hip_atomic_load(grp + 64 + lane, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return __builtin_bit_cast(T, w);
}
__device__ __forceinline__ void sum_put_f(float *p, float x)
{
    __hip_atomic_store((unsigned int *)p, __float_as_uint(x), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float sum_get_f(const float *p)
{
    return __uint_as_float(
        __hip_atomic_load((const unsigned int *)p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
}

template <int HALF>
__device__ __forceinline__ h8 set_half(h8 x, h4 r)
{
    if constexpr (HALF == 0) return h8{r[0], r[1], r[2], r[3], x[4], x[5], x[6], x[7]};
    else return h8{x[0], x[1], x[2], x[3], r[0], r[1], r[2], r[3]};
}
// DV = false: the forward O = F / G.  DV = true: the reverse-causal
// numerator of the backward, dv_n = sum_{i >= n} f(k^_n . q^_i) u_i with
// u_i = dO_i / G_i (Sec. 2.5): the scan runs over the tokens in reverse order
// (logical token n is row N-1-n), q and k trade roles (the caller passes k^ as
// q and q^ as k, both already standardised, in fp16), v is dO scaled per row
// by rg = 1/G, and F is stored without the divide; the denominator terms are
// skipped.
// One workgroup of the scan: block b (the scan's own numbering; when the
// scan shares a launch with other work, b counts from its first block, whose
// id must be a multiple of 8 for the XCD mapping below).  Blocks
// [0, nitems) are the (head, slice) items (their first segments when the
// scan is split), blocks [nitems, 2 nitems) their second segments.
template <bool DV>
__device__ __forceinline__ void scan_block(Smem &sm, const _Float16 *__restrict__ q,
                                           const _Float16 *__restrict__ k,
                                           const bf16_t *__restrict__ v, bf16_t *__restrict__ out,
                                           float *__restrict__ g, const float *__restrict__ rg,
                                           int N, int BH, int b, int nitems, const SegArgs &sa)
{
    int seg = 0;
    if (sa.split && b >= nitems) {
        seg = 1;
        b -= nitems;
    }
    const int item = b;
    // XCD-aware mapping: consecutive block ids land on different XCDs
    // (round-robin over 8); keep the 4 slices of a head on one XCD so that
    // its q and k rows are shared through that XCD's L2.
    int head, sl;
    if ((nitems & 31) == 0) {
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

    // max |v| over this slice -> power-of-two scale (eight loads in flight
    // per thread, not one round trip per row pair)
    {
        const int tid = threadIdx.x;
        float vmax = 0.f;
        constexpr int U = 8;
        for (int p0 = tid; p0 < 2 * N; p0 += U * NTH) {
            uint4 raw[U];
            float rr[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int p = p0 + u * NTH, n = p >> 1, hh = p & 1;
                raw[u] = uint4{0u, 0u, 0u, 0u};
                rr[u] = 0.0f;
                if (p < 2 * N) {
                    raw[u] = *(const uint4 *)(v + (size_t)n * D + SL * sl + 8 * hh);
                    // raw: no arithmetic on a loaded value before all U are issued
                    rr[u] = DV ? rg[n] : 1.0f;
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
        if (tid < D) sm.y2[0][tid] = sm.y2s[0][tid] = 0.f;
        if (tid < SL) sm.x1[0][tid] = 0.f;
        for (int e = tid; e < D * RS64; e += NTH) sm.y3h[e] = (_Float16)0.0f;
    }
    __syncthreads();
    float vmax = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) vmax = fmaxf(vmax, sm.red[w]);
    const int vexp = pow2_exponent(vmax * 63.0f * (float)N);
    const float vscale = ldexpf(1.0f, -vexp);   // v -> v * 2^-e
    const float oscale = ldexpf(1.0f, vexp);
    const int nch = (N + C - 1) / C;

    // chunk range of this workgroup; [cstart, cbeg) are build-only chunks
    // (a second segment rebuilding its prefix)
    const int cbeg = seg ? sa.csplit : 0;
    const int cend = (sa.split && seg == 0) ? sa.csplit : nch;
    int cstart = cbeg;
    bool loaded = false;
    unsigned char *sum = sa.split ? sa.sum + (size_t)item * SUM_BYTES : nullptr;
    if (seg == 1) {
        if (sa.wait) {
            // one thread polls; the summary loads (sum_get) come after the
            // barrier that follows
            if (threadIdx.x == 0) {
                unsigned int f = 0;
                for (int it = 0; it < SEG_SPIN; ++it) {
                    f = __hip_atomic_load(sa.flags + item, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    if (f) break;
                    __builtin_amdgcn_s_sleep(8);
                }
                sm.segok = f != 0;
            }
            __syncthreads();
            loaded = sm.segok != 0;
        }
        if (!loaded) cstart = 0;
    }
    // summary groups of 64 lanes x 16 bytes: state (wave, pair), Y3 (helper, tile)
    unsigned long long *sum_ast = (unsigned long long *)sum;
    unsigned long long *sum_y3 = (unsigned long long *)(sum + SUM_AST);
    float *sum_misc = (float *)(sum + SUM_AST + SUM_Y3);

    const int w = threadIdx.x >> 6;
    const bool is_state = w < NSW;
    const int hw = w - NSW;   // helper index

    // Lane-derived LDS offsets are recomputed in every phase from an opaque
    // copy of the thread id: hoisted out of the loop they would stay live for
    // the whole scan.
    int tid = threadIdx.x;
    int lane = tid & 63, r16 = lane & 15, h = lane >> 4;
    auto refresh_ids = [&]() {
        asm volatile("" : "+v"(tid));
        lane = tid & 63;
        r16 = lane & 15;
        h = lane >> 4;
    };

    // The two roles run separate loops with the same barrier sequence (one
    // after staging chunk 0, two per chunk); the role is uniform per wave.
    if (is_state) {
        // fp16 state, paired per query K step
        h8 Ast[NKS];
#pragma unroll
        for (int p = 0; p < NKS; ++p)
            Ast[p] = loaded ? sum_get_lane<h8>(sum_ast + (w * NKS + p) * 128, lane)
                            : h8{0, 0, 0, 0, 0, 0, 0, 0};
        __syncthreads();
        for (int c = cstart; c < cend; ++c) {
            // ---- (1) query contraction over the wave's tiles, 128 tokens ----
            __builtin_amdgcn_sched_barrier(0);
            refresh_ids();
            const bool build = c < cbeg;
            // the q^ values of a row tile: l blocks, the linear tile and the
            // wave's channels; loaded one row tile ahead of their use
            struct QRow {
                h4 myl[4], mylin;
                h4 qc[4];
            };
            auto loadq = [&](int rt, QRow &r) {
                const int tok = 16 * rt + r16;
#pragma unroll
                for (int u = 0; u < 4; ++u) r.myl[u] = ld4(sm.qrow + sw64(tok, 16 * u + 4 * h));
                r.mylin = ld4(sm.qrow + sw64(tok, 16 * w + 4 * h));
#pragma unroll
                for (int a = 0; a < 4; ++a) r.qc[a] = ld4(sm.qrow + sw64(tok, 16 * a + 4 * w));
            };
            auto contract = [&](int rt, const QRow &r) {
                const int tok = 16 * rt + r16;
                f4 F0 = {0.f, 0.f, 0.f, 0.f}, F1 = {0.f, 0.f, 0.f, 0.f};
                auto gen = [&](auto ti) -> h4 {
                    constexpr int t = decltype(ti)::value;
                    constexpr Tile T = tile_of(t < NT ? t : 0);
                    if constexpr (t >= NT) {
                        return h4{0, 0, 0, 0};
                    } else if constexpr (T.kind == 0) {
                        return r.mylin;
                    } else {
                        const _Float16 qm = r.qc[T.i / 4][T.i % 4];
                        return scale4(r.myl[T.u], qm);
                    }
                };
                static_for<0, NKS>([&](auto pi) {
                    constexpr int p = decltype(pi)::value;
                    const h8 B = cat(gen(std::integral_constant<int, 2 * p>{}),
                                     gen(std::integral_constant<int, 2 * p + 1>{}));
                    if constexpr (p & 1) F1 = mfma(Ast[p], B, F1);
                    else F0 = mfma(Ast[p], B, F0);
                });
                *(f4 *)(sm.fpart + ((w * 4 + h) * C + tok) * 4) = F0 + F1;
            };
            if (!build) {
                QRow ra, rb;
                loadq(0, ra);
#pragma unroll 1
                for (int rt = 0; rt < NRT; rt += 2) {
                    loadq(rt + 1, rb);
                    contract(rt, ra);
                    if (rt + 2 < NRT) loadq(rt + 2, ra);
                    contract(rt + 1, rb);
                }
            }
            __syncthreads();

            // ---- (2) state update S += Phi(K)^T V (Sec. 2.4) ----------------
            __builtin_amdgcn_sched_barrier(0);
            refresh_ids();
            const _Float16 *kTc = sm.kT[c & 1];
            const _Float16 *vTc = sm.vT[c & 1];
            h8 Ak[4][NKS2];
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int s = 0; s < NKS2; ++s) Ak[u][s] = ld8(kTc + sw128(16 * u + r16, 32 * s + 8 * h));
            h8 Vf[NKS2];
#pragma unroll
            for (int s = 0; s < NKS2; ++s) Vf[s] = ld8(vTc + sw128(r16, 32 * s + 8 * h));
            {
                // linear tile: x2[l][j] += sum_t k_tl v_tj, l in tile w
                f4 acc = mfma(ld8(kTc + sw128(16 * w + r16, 8 * h)), Vf[0], f4{0.f, 0.f, 0.f, 0.f});
#pragma unroll
                for (int s = 1; s < NKS2; ++s)
                    acc = mfma(ld8(kTc + sw128(16 * w + r16, 32 * s + 8 * h)), Vf[s], acc);
                const h8 cur = Ast[0];
                Ast[0] = set_half<0>(Ast[0], cvt4(acc) + h4{cur[0], cur[1], cur[2], cur[3]});
            }
            static_for<0, NQ>([&](auto ii) {
                constexpr int i = decltype(ii)::value;
                constexpr int u0 = u0_of(i);
                constexpr int t0 = first_tile(i);
                constexpr int nu = 4 - u0;
                const int m = 16 * u0 + 4 * w + (i & 3);
                h8 Wm[NKS2];
#pragma unroll
                for (int s = 0; s < NKS2; ++s) Wm[s] = ld8(kTc + sw128(m, 32 * s + 8 * h)) * Vf[s];
                // the chunk's contribution from zero, rounded to fp16 and added
                // to the fp16 state with packed fp16 arithmetic (the diagonal
                // tile, stored halved, takes half the contribution)
                f4 acc[nu];
                static_for<0, nu>([&](auto ui) {
                    constexpr int uu = decltype(ui)::value;
                    acc[uu] = mfma(Ak[u0 + uu][0], Wm[0], f4{0.f, 0.f, 0.f, 0.f});
                });
#pragma unroll
                for (int s = 1; s < NKS2; ++s)
                    static_for<0, nu>([&](auto ui) {
                        constexpr int uu = decltype(ui)::value;
                        acc[uu] = mfma(Ak[u0 + uu][s], Wm[s], acc[uu]);
                    });
                static_for<0, nu>([&](auto ui) {
                    constexpr int uu = decltype(ui)::value;
                    constexpr int t = t0 + uu;
                    h4 a16 = cvt4(acc[uu]);
                    if constexpr (uu == 0) a16 = a16 * (_Float16)0.5f;
                    // in place on the whole pair (the other half adds zero)
                    const h4 z4 = {0, 0, 0, 0};
                    Ast[t / 2] = Ast[t / 2] + ((t & 1) ? cat(z4, a16) : cat(a16, z4));
                });
            });
            __syncthreads();
        }
        if (sum && seg == 0) {
#pragma unroll
            for (int p = 0; p < NKS; ++p)
                sum_put_lane(sum_ast + (w * NKS + p) * 128, threadIdx.x & 63, Ast[p]);
        }
    } else {
        // loader roles: tokens 4*tg .. 4*tg+3, channels 8*cg .. 8*cg+7; v:
        // token vt, columns 8*vh .. 8*vh+7
        uint4 pq[4], pk[4], pv;
        float prg = 1.0f;
        f4 y3acc[3] = {f4{0.f, 0.f, 0.f, 0.f}, f4{0.f, 0.f, 0.f, 0.f}, f4{0.f, 0.f, 0.f, 0.f}};
        // Y3 in LDS is Y3 * 2^-gexp, gexp fixed by the tokens summed so far
        int gexp = loaded ? max(0, pow2_exponent(64.0f * (float)(cbeg * C))) : 0;
        if (loaded) {
#pragma unroll
            for (int kk = 0; kk < 3; ++kk) y3acc[kk] = sum_get_lane<f4>(sum_y3 + (hw * 3 + kk) * 128, lane);
        }
        const h8 ones8 = {1, 1, 1, 1, 1, 1, 1, 1};
        // the scaled fp16 copy of this helper's Y3 tile kk (Y3[m][l] and, off
        // the diagonal, Y3[l][m])
        auto put_y3h = [&](int kk, float gs) {
            int u, u2;
            y3_tile(hw, kk, u, u2);
            // lane: column m = 16*u2 + r16, rows l = 16*u + 4h + i
            const int mcol = 16 * u2 + r16;
            h4 hv;
#pragma unroll
            for (int i = 0; i < 4; ++i) hv[i] = (_Float16)(y3acc[kk][i] * gs);
            *(h4 *)(sm.y3h + sw64(mcol, 16 * u + 4 * h)) = hv;   // Y3[m][l]
            if (u != u2) {
#pragma unroll
                for (int i = 0; i < 4; ++i) sm.y3h[sw64(16 * u + 4 * h + i, mcol)] = hv[i];
            }
        };

        auto prefetch = [&](int c) {
            const int ht = tid - NSW * 64;
            const int tg = ht >> 3, cg = ht & 7;
            const uint4 z = {0u, 0u, 0u, 0u};
            const int nb = c * C + 4 * tg;
            if (nb + 3 < N) {
                // all four rows in range (every chunk but the last): one base
                // address, the rows at fixed offsets from it
                constexpr int step = DV ? -D : D;
                const size_t p0 = DV ? (size_t)(N - 1 - nb) : (size_t)nb;
                const _Float16 *qp = q + p0 * D + 8 * cg, *kp = k + p0 * D + 8 * cg;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    pq[j] = *(const uint4 *)(qp + j * step);
                    pk[j] = *(const uint4 *)(kp + j * step);
                }
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int n = nb + j;
                    pq[j] = pk[j] = z;
                    if (n < N) {
                        const size_t pn = DV ? (size_t)(N - 1 - n) : (size_t)n;
                        pq[j] = *(const uint4 *)(q + pn * D + 8 * cg);
                        pk[j] = *(const uint4 *)(k + pn * D + 8 * cg);
                    }
                }
            }
            const int vt = ht >> 1, vh = ht & 1;
            const int nv = c * C + vt;
            pv = z;
            if (nv < N) {
                const size_t pn = DV ? (size_t)(N - 1 - nv) : (size_t)nv;
                pv = *(const uint4 *)(v + pn * D + SL * sl + 8 * vh);
                if constexpr (DV) prg = rg[pn];
            }
        };
        // Staging of chunk c: store q^ (row-major), k^
        // (row-major and transposed) and the scaled v transposed.  q^, k^
        // arrive standardised (Sec. 2.2, Eqs. 6-7) in fp16; rows past N are
        // zero.
        auto stage = [&](int c) {
            const int ht = tid - NSW * 64;
            const int tg = ht >> 3, cg = ht & 7;
            const int buf = c & 1;
            h8 hk[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int row = 4 * tg + j;
                const h8 hq = __builtin_bit_cast(h8, pq[j]);
                *(h8 *)(sm.qrow + sw64(row, 8 * cg)) = hq;
                hk[j] = __builtin_bit_cast(h8, pk[j]);
                *(h8 *)(sm.krow + sw64(row, 8 * cg)) = hk[j];
            }
#pragma unroll
            for (int i = 0; i < 8; ++i)
                *(h4 *)(sm.kT[buf] + sw128(8 * cg + i, 4 * tg)) =
                    h4{hk[0][i], hk[1][i], hk[2][i], hk[3][i]};
            const int vt = ht >> 1, vh = ht & 1;
            float xv[8];
            bf16x8_to_f32(pv, xv);
            const float vs = DV ? vscale * prg : vscale;
#pragma unroll
            for (int i = 0; i < 8; ++i) sm.vT[buf][sw128(8 * vh + i, vt)] = (_Float16)(xv[i] * vs);
        };

        prefetch(cstart);
        stage(cstart);
        if (loaded) {
            // segment 0's prefix sums, as its last chunk left them in LDS
            const int ht = tid - NSW * 64, cb = cbeg & 1;
            if (!DV && ht < D) {
                sm.y2[cb][ht] = sum_get_f(sum_misc + ht);
                sm.y2s[cb][ht] = sum_get_f(sum_misc + D + ht);
            }
            if (ht < SL) sm.x1[cb][ht] = sum_get_f(sum_misc + 2 * D + ht);
            if (!DV) {
                const int ny3 = y3_count(hw);
                const float gs = ldexpf(1.0f, -gexp);
#pragma unroll
                for (int kk = 0; kk < 3; ++kk)
                    if (kk < ny3) put_y3h(kk, gs);
            }
        }
        __syncthreads();
        for (int c = cstart; c < cend; ++c) {
            const int n0 = c * C;
            const int nvalid = min(C, N - n0);
            const int cur = c & 1, nxt = cur ^ 1;
            const bool more = c + 1 < cend;
            const bool build = c < cbeg;   // prefix only: no outputs

            // ---- (1) in-chunk block and denominators, row tiles hw, 7 - hw
            //      (1 + 4, 1 + 4, 2 + 3, 2 + 3 tile-pair items) ---------------
            __builtin_amdgcn_sched_barrier(0);
            refresh_ids();
            if (more) prefetch(c + 1);
            f4 Fin[2];
            float Gs[2];
            if (!build) {
                const _Float16 *vTc = sm.vT[cur];
#pragma unroll
                for (int r = 0; r < 2; ++r) {
                    const int rt = r ? NRT - 1 - hw : hw;
                    const int tok = 16 * rt + r16;
                    const h8 QB0 = ld8(sm.qrow + sw64(tok, 8 * h));
                    const h8 QB1 = ld8(sm.qrow + sw64(tok, 32 + 8 * h));
                    f4 F = {0.f, 0.f, 0.f, 0.f};
                    // in-chunk row sums of the weights: every row of
                    // ones x W is the column sum, so each lane holds the full
                    // sum for its query
                    f4 Gin = {0.f, 0.f, 0.f, 0.f};
                    // S^T tile (rows: keys 16tt.., columns: queries) -> 2 f(s):
                    // the accumulator starts at 1, so t = s + 1 and
                    // 2 f_2(s) = t^2 + 1 is one FMA; the factor 2 is removed
                    // where F and G are combined
                    auto wtile = [&](int tt, bool diag) -> h4 {
                        f4 S = {1.f, 1.f, 1.f, 1.f};
                        S = mfma(ld8(sm.krow + sw64(16 * tt + r16, 8 * h)), QB0, S);
                        S = mfma(ld8(sm.krow + sw64(16 * tt + r16, 32 + 8 * h)), QB1, S);
                        f4 wv;
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            float y = fmaf(S[i], S[i], 1.0f);
                            if (diag && (4 * h + i) > r16) y = 0.0f;
                            wv[i] = y;
                        }
                        return cvt4(wv);
                    };
                    // whole tile pairs below the diagonal tile
#pragma unroll 1
                    for (int j = 0; j < rt / 2; ++j) {
                        const int a = 2 * j;
                        const h4 wa = wtile(a, false), wb = wtile(a + 1, false);
                        F = mfma(cat(ld4(vTc + sw128(r16, 16 * a + 4 * h)),
                                     ld4(vTc + sw128(r16, 16 * a + 16 + 4 * h))),
                                 cat(wa, wb), F);
                        if constexpr (!DV) Gin = mfma(ones8, cat(wa, wb), Gin);
                    }
                    {
                        // the last pair holds the diagonal tile rt (masked to
                        // keys <= query), alone when rt is even
                        const int a = rt & ~1;
                        const h4 wa = wtile(a, a == rt);
                        const h4 va = ld4(vTc + sw128(r16, 16 * a + 4 * h));
                        h4 wb = h4{0, 0, 0, 0}, vb = h4{0, 0, 0, 0};
                        if (a != rt) {
                            wb = wtile(rt, true);
                            vb = ld4(vTc + sw128(r16, 16 * rt + 4 * h));
                        }
                        F = mfma(cat(va, vb), cat(wa, wb), F);
                        if constexpr (!DV) Gin = mfma(ones8, cat(wa, wb), Gin);
                    }
                    float gpart = 0.f;
                    if (!DV) {
                        // inter-chunk denominator q.y2 + 1/2 q^T Y3 q (+ n0)
                        float gq = 0.f;
#pragma unroll
                        for (int cc = 0; cc < 4; ++cc) {
                            const h4 ql = ld4(sm.qrow + sw64(tok, 16 * cc + 4 * h));
                            f4 T = *(const f4 *)(sm.y2s[cur] + 16 * cc + 4 * h);
                            T = mfma(ld8(sm.y3h + sw64(16 * cc + r16, 8 * h)), QB0, T);
                            T = mfma(ld8(sm.y3h + sw64(16 * cc + r16, 32 + 8 * h)), QB1, T);
#pragma unroll
                            for (int i = 0; i < 4; ++i) gq = fmaf((float)ql[i], T[i], gq);
                        }
                        gpart = fmaf(0.5f * ldexpf(1.0f, gexp), gq, gpart);
                        if (h == 0) gpart += (float)n0;
                    }
                    gpart = rows4_sum(gpart);
                    gpart = fmaf(0.5f, Gin[0], gpart);
                    Fin[r] = F;
                    Gs[r] = gpart;
                }
            }
            __syncthreads();

            // ---- (2) output, prefix sums, Y3, staging of the next chunk ------
            __builtin_amdgcn_sched_barrier(0);
            refresh_ids();
            const _Float16 *kTc = sm.kT[cur];
            const _Float16 *vTc = sm.vT[cur];
#pragma unroll
            for (int r = 0; r < 2; ++r) {
                if (build) break;
                const int rt = r ? NRT - 1 - hw : hw;
                const int tok = 16 * rt + r16;
                f4 F = 0.5f * Fin[r] + *(const f4 *)(sm.x1[cur] + 4 * h);
#pragma unroll
                for (int ww = 0; ww < NSW; ++ww)
                    F += *(const f4 *)(sm.fpart + ((ww * 4 + h) * C + tok) * 4);
                if (n0 + tok < N) {
                    const float sc = DV ? oscale : oscale * __builtin_amdgcn_rcpf(Gs[r]);
                    uint2 o;
                    o.x = pack_bf16x2(F[0] * sc, F[1] * sc);
                    o.y = pack_bf16x2(F[2] * sc, F[3] * sc);
                    const size_t pn = DV ? (size_t)(N - 1 - (n0 + tok)) : (size_t)(n0 + tok);
                    *(uint2 *)(out + pn * D + SL * sl + 4 * h) = o;
                    if (!DV && g && sl == 0 && h == 0) g[n0 + tok] = Gs[r];
                }
            }
            // prefix sums y2 (channels 16hw..16hw+15) and x1 (helper 0) as
            // row sums (k^T or v^T) x ones: lane (r16, h) holds the sums of
            // rows 4h..4h+3
            const int gnext = max(0, pow2_exponent(64.0f * (float)(n0 + nvalid)));
            if (!DV) {
                f4 s4 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int st = 0; st < NKS2; ++st)
                    s4 = mfma(ld8(kTc + sw128(16 * hw + r16, 32 * st + 8 * h)), ones8, s4);
                if (r16 == 0) {
                    const f4 y = *(const f4 *)(sm.y2[cur] + 16 * hw + 4 * h) + s4;
                    *(f4 *)(sm.y2[nxt] + 16 * hw + 4 * h) = y;
                    *(f4 *)(sm.y2s[nxt] + 16 * hw + 4 * h) = ldexpf(2.0f, -gnext) * y;
                }
            }
            if (hw == 0) {
                f4 s4 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int st = 0; st < NKS2; ++st)
                    s4 = mfma(ld8(vTc + sw128(r16, 32 * st + 8 * h)), ones8, s4);
                if (r16 == 0) *(f4 *)(sm.x1[nxt] + 4 * h) = *(const f4 *)(sm.x1[cur] + 4 * h) + s4;
            }
            if (!DV) {
                // Y3 += K^T K and its scaled fp16 copy for the next chunk
                const int ny3 = y3_count(hw);
                const float gs = ldexpf(1.0f, -gnext);
#pragma unroll
                for (int kk = 0; kk < 3; ++kk) {
                    if (kk >= ny3) break;
                    int u, u2;
                    y3_tile(hw, kk, u, u2);
#pragma unroll
                    for (int s = 0; s < NKS2; ++s)
                        y3acc[kk] = mfma(ld8(kTc + sw128(16 * u + r16, 32 * s + 8 * h)),
                                         ld8(kTc + sw128(16 * u2 + r16, 32 * s + 8 * h)), y3acc[kk]);
                    put_y3h(kk, gs);
                }
                gexp = gnext;
            }
            if (more) stage(c + 1);
            __syncthreads();
        }
        if (sum && seg == 0) {
            // the summary: Y3 accumulators and the prefix sums after the last chunk
            const int ln = threadIdx.x & 63, ht = threadIdx.x - NSW * 64, cb = cend & 1;
#pragma unroll
            for (int kk = 0; kk < 3; ++kk) sum_put_lane(sum_y3 + (hw * 3 + kk) * 128, ln, y3acc[kk]);
            if (!DV && ht < D) {
                sum_put_f(sum_misc + ht, sm.y2[cb][ht]);
                sum_put_f(sum_misc + D + ht, sm.y2s[cb][ht]);
            }
            if (ht < SL) sum_put_f(sum_misc + 2 * D + ht, sm.x1[cb][ht]);
        }
    }
    if (sum && seg == 0) {
        // publish: every thread's summary stores have completed (waitcnt on
        // all counters) before the barrier, the flag goes up after it
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        if (threadIdx.x == 0)
            __hip_atomic_store(sa.flags + item, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

}  // namespace mfma_causal
}  // namespace fm

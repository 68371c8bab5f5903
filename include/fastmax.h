/*
 * fastmax.h -- C ABI of the MI355X (gfx950) Fastmax attention library.
 *
 * Fastmax (Gerami, Hoover, Dulepet, Duraiswami, "FAST: Factorizable Attention
 * for Speeding up Transformers", arXiv 2402.07901) computes, per head,
 *
 *     q^_i = (q_i - mean q_i) / std(q_i - mean q_i)       (Sec. 2.2, Eqs. 6-7)
 *     k^_n likewise
 *     s_in = q^_i . k^_n,   w_in = f_p(s_in) = sum_{l<=p} s_in^l / l!
 *                                                    (Sec. 2.2, Eq. "taylor")
 *     G_i  = sum_n w_in,    F_i = sum_n w_in v_n,    O_i = F_i / G_i
 *                                     (Sec. 2.2 a_ij, Eq. "tobeexpanded";
 *                                      Sec. 2.4 Eq. "bigo")
 *
 * with n running over all N tokens, or over n <= i when causal (Sec. 2.1
 * tril mask; Sec. 2.4 causal F and G).  The library evaluates it exactly
 * through the factorisation of Sec. 2.4 (moments of k^ and v contracted
 * against powers of q^), never forming the N x N matrix.
 *
 * Conventions shared by every entry point
 *  - Layout: q, k, v, out, dout, dq, dk, dv are [B, H, N, D] contiguous
 *    (D fastest) in the I/O dtype `dt`; g is [B, H, N] float32.
 *    Statistics (standardisation, G) are float32 whatever `dt` is; moment
 *    contractions accumulate in float32.  The causal bf16, D = 64, p = 2
 *    MFMA path carries its moment state between 128-token chunks in fp16
 *    (each chunk's float32 contribution is rounded and added); its error
 *    stays within the bf16 tolerance on every row of 65536-token causal
 *    sequences (tested).
 *  - Pointers are device pointers (HBM) and must be 16-byte aligned.
 *  - Ownership: the caller owns every buffer, including `workspace`.  The
 *    library keeps no pointer after return, allocates no device memory,
 *    creates no stream and holds no global mutable state (thread-safe);
 *    the exceptions are fastmax_fwd_noalloc's per-GPU scratch array and the
 *    process-wide mode of fastmax_set_scan_segments.
 *  - Device: the kernels run on the device that is current at the call;
 *    `stream`, if not 0, must belong to it (FASTMAX_EINVAL otherwise).
 *  - Asynchrony: work is enqueued on `stream` (0 = the null stream);
 *    FASTMAX_OK means "enqueued".  Outputs are valid once the stream reaches
 *    that point.  Inputs must stay valid until then.
 *  - Validation happens on the host before anything is enqueued (the only
 *    HIP calls before it ask which device is current and which device the
 *    stream belongs to): on any error nothing is enqueued and nothing is
 *    written.
 *  - Supported: D in {16, 32, 64, 128} (fp16 MFMA kernels serve D = 64,
 *    p = 2, bf16, except non-causal below 128 tokens; every other case runs
 *    on float32 MFMA kernels, and the dropout calls on float32 VALU kernels);
 *    p in {1, 2}; causal in {0, 1};
 *    dt in {FASTMAX_F32, FASTMAX_BF16}; B, H, N >= 1, B*H <= 2^20 heads,
 *    N <= 2^30 tokens per head and B*H*N*D < 2^62.
 *  - A token whose q or k row is constant has std 0; its standardised row is
 *    undefined (as in the paper) and its outputs are not finite.
 *  - Errors are reported only through the return code (nothing printed).
 */
#ifndef FASTMAX_H
#define FASTMAX_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    FASTMAX_F32 = 0,  /* float32 I/O  */
    FASTMAX_BF16 = 1  /* bfloat16 I/O (round-to-nearest-even on output) */
} fastmax_dtype_t;

enum {
    FASTMAX_OK = 0,
    FASTMAX_EINVAL = -1,       /* p, causal, dt, qk_scale or dropout rate out of range; B, H or N
                                  < 1, or beyond the size limits above; a stream of another
                                  device */
    FASTMAX_EUNSUPPORTED = -2, /* head dimension D not in {16, 32, 64, 128}, or a call
                                  whose launch grids would exceed the dispatch limits
                                  (2^32 - 1 work-items per grid dimension; only at extreme
                                  head counts, e.g. 2^18 heads at D = 128, p = 2, or 2^20
                                  in the bf16 D = 64 backward); nothing is enqueued */
    FASTMAX_ENULL = -3,        /* a required pointer is NULL                  */
    FASTMAX_EALIGN = -4,       /* a tensor pointer is not 16-byte aligned     */
    FASTMAX_EWORKSPACE = -5,   /* workspace NULL or smaller than required     */
    FASTMAX_EHIP = -6          /* the HIP runtime rejected a launch           */
};

/*
 * Bytes of device workspace fastmax_fwd (backward = 0) or fastmax_bwd
 * (backward = 1) needs for this problem.  0 means no workspace is needed
 * (NULL may then be passed).  Returns 0 as well for arguments the entry
 * point would reject in its argument checks (EINVAL, EUNSUPPORTED for D); a
 * call refused for its launch grids (EUNSUPPORTED at extreme head counts)
 * still gets its size here.  The workspace need not be zeroed.  The forward needs
 * one when it splits each head's sequence into segments whose moment states
 * are built in parallel: the non-causal bf16, D = 64, p = 2 path with
 * N >= 128 (per-segment partial moments, their fp16 sum and the per-head
 * denominator terms, about 0.7 MB per (head, segment)), and every other
 * non-MFMA forward when B*H is small (fp32 segment states, enough segments
 * for about 256 workgroups).  The causal bf16, D = 64, p = 2 forward keeps
 * the standardised q and k in fp16 (256 bytes per row) and, for N > 128,
 * room for the summaries of split scans (99072 bytes per head and 16-column
 * slice, see fastmax_set_scan_segments).  The backward always
 * needs one: per token 1/G, c = dO.O/G, the fp32
 * gradient accumulators of q^ and k^ and (causal bf16, D = 64, p = 2) the
 * standardised q^, k^ in fp16, the dv scan's segment summaries, plus
 * per-chunk maxima; on the float32 path
 * with few heads (B*H times the column slices under about 256) also the
 * per-segment moment states of its two scans.
 */
size_t fastmax_workspace_bytes(int B, int H, int N, int D, int p, int causal,
                               fastmax_dtype_t dt, int backward);

/*
 * Forward pass (Sec. 2.2 definition; evaluated by the Sec. 2.4 factorisation,
 * with the causal moments carried across chunks of tokens).
 *   q, k, v : inputs  [B, H, N, D] in dt
 *   out     : output  [B, H, N, D] in dt, O = F / G
 *   g       : optional output [B, H, N] float32, G_i = sum_n f_p(s_in)
 *             (the row sums the backward needs, Sec. 2.5); NULL to skip.
 * Returns FASTMAX_OK or a negative FASTMAX_E* code.
 */
int fastmax_fwd(const void *q, const void *k, const void *v, void *out,
                float *g, int B, int H, int N, int D, int p, int causal,
                fastmax_dtype_t dt, void *workspace, size_t workspace_bytes,
                hipStream_t stream);

/*
 * Backward pass: gradients of sum(dout * O) with respect to q, k and v,
 * following the score derivative of Sec. 2.3 (Eq. "bound", read with
 * a_in / a_il) and the custom-gradient idea of Sec. 2.5: only O and G are
 * saved from the forward; q^, k^ are recomputed and every N x N quantity is
 * replaced by moment contractions.
 *   q, k, v : forward inputs            [B, H, N, D] in dt
 *   out     : forward output O          [B, H, N, D] in dt
 *   dout    : upstream gradient dL/dO   [B, H, N, D] in dt
 *   g       : forward row sums G        [B, H, N] float32 (from fastmax_fwd)
 *   dq, dk, dv : outputs                [B, H, N, D] in dt
 * The same (p, causal) as the forward must be passed.
 */
int fastmax_bwd(const void *q, const void *k, const void *v, const void *out,
                const void *dout, const float *g, void *dq, void *dk, void *dv,
                int B, int H, int N, int D, int p, int causal,
                fastmax_dtype_t dt, void *workspace, size_t workspace_bytes,
                hipStream_t stream);

/*
 * Score-scaled variants: the weights become f_p(qk_scale * q^.k^).  The
 * paper's definition (Sec. 2.2) has no temperature, which is qk_scale = 1
 * (fastmax_fwd and fastmax_bwd are these calls with 1).  qk_scale = 1/D is
 * the unit-norm variant (q^ and k^ divided by sqrt(D)), under which
 * |qk_scale * s| <= 1 as the bound of Sec. 2.3 assumes, so f_1 >= 0 and the
 * rows of the attention matrix are convex weights (Eq. "valid"); 1/sqrt(D)
 * is softmax's temperature (Sec. 2.1).  qk_scale must lie in (0, 1], else
 * FASTMAX_EINVAL.  Arguments, layouts, workspace and errors are otherwise
 * those of fastmax_fwd and fastmax_bwd (the workspace size does not depend
 * on qk_scale); the backward must be given the forward's qk_scale.
 */
int fastmax_fwd_scaled(const void *q, const void *k, const void *v, void *out,
                       float *g, int B, int H, int N, int D, int p, int causal,
                       float qk_scale, fastmax_dtype_t dt, void *workspace,
                       size_t workspace_bytes, hipStream_t stream);
int fastmax_bwd_scaled(const void *q, const void *k, const void *v, const void *out,
                       const void *dout, const float *g, void *dq, void *dk, void *dv,
                       int B, int H, int N, int D, int p, int causal, float qk_scale,
                       fastmax_dtype_t dt, void *workspace, size_t workspace_bytes,
                       hipStream_t stream);

/* Static description of a return code (never NULL). */
/*
 * Quadratic-term dropout, for training (Sec. 2.4, the dropout paragraph, and
 * Fig. 2, whose "quadratic" variant is the one built here).  Only p = 2.
 * Every key token n carries a keep bit for each of its D(D+1)/2 quadratic
 * features k^_nm k^_nl (m <= l, numbered m-major: t = m D - m(m-1)/2 + l - m).
 * A kept feature is multiplied by 1/(1 - rate), a dropped one by 0, in both
 * the numerator and the denominator moments (it is one embedding), so the
 * weight of the pair (i, n) becomes
 *     w_in = 1 + tau s_in + sum_{m<=l} c_ml tau^2 q^_im q^_il k^_nm k^_nl b~_nt
 * (c_mm = 1/2, c_ml = 1 for m < l, b~ = bit / (1 - rate)); O = F / G as before.
 * With every bit set and rate 0 this is the plain p = 2 forward.
 *
 * keep_bits: uint32 [B, H, N, fastmax_dropout_mask_words(D)], 4-byte aligned,
 *   feature t of token n at bit t % 32 of word t / 32 of the token's row
 *   (bits past D(D+1)/2 are ignored).  The caller owns it and passes the same
 *   bits to the forward and the backward of one step.
 * The dropout calls run on the float32 VALU kernels for every D and dtype.
 */

/* Words per token of a keep-bit row: ceil(D(D+1)/2 / 32); 0 for an
 * unsupported D. */
size_t fastmax_dropout_mask_words(int D);

/*
 * Draws keep bits with the counter-based generator Philox4x32-10 (Salmon,
 * Moraes, Dror, Shaw, "Parallel Random Numbers: As Easy as 1, 2, 3", SC 2011):
 * for head h = b H + head index and token n, feature t uses output word t % 4
 * of the counter (n, t / 4, h, 0) under the key (seed & 0xffffffff,
 * seed >> 32) and is kept iff that word is >= floor(rate 2^32).  Writes every
 * word of keep_bits (padding bits 0).  Same seed, same bits, on any device.
 * rate in [0, 1); EINVAL otherwise.
 */
int fastmax_dropout_mask(uint32_t *keep_bits, int B, int H, int N, int D, float rate,
                         uint64_t seed, hipStream_t stream);

/* Workspace of fastmax_fwd_dropout (backward = 0) / fastmax_bwd_dropout
 * (backward = 1): that of the float32 kernels at p = 2 (see
 * fastmax_workspace_bytes) and, for the causal forward, after it (rounded up
 * to 256 bytes) the masked in-chunk weights: 16 x 16 floats per chunk of 16
 * tokens of every head (64 bytes per token).  Returns 0 for arguments the
 * entry points would reject. */
size_t fastmax_dropout_workspace_bytes(int B, int H, int N, int D, int causal,
                                       fastmax_dtype_t dt, int backward);

/* Forward with the masked weights.  Arguments as fastmax_fwd_scaled with
 * p = 2, plus keep_bits and rate (the drop probability the bits were drawn
 * with; kept features are scaled by 1/(1 - rate)).  g receives G of the
 * masked weights. */
int fastmax_fwd_dropout(const void *q, const void *k, const void *v, void *out, float *g,
                        const uint32_t *keep_bits, float rate, int B, int H, int N, int D,
                        int causal, float qk_scale, fastmax_dtype_t dt, void *workspace,
                        size_t workspace_bytes, hipStream_t stream);

/* Backward of fastmax_fwd_dropout with the same keep_bits and rate (the
 * mask is a constant of the step): out and g are that forward's outputs.
 * Arguments as fastmax_bwd_scaled with p = 2. */
int fastmax_bwd_dropout(const void *q, const void *k, const void *v, const void *out,
                        const void *dout, const float *g, const uint32_t *keep_bits, float rate,
                        void *dq, void *dk, void *dv, int B, int H, int N, int D, int causal,
                        float qk_scale, fastmax_dtype_t dt, void *workspace,
                        size_t workspace_bytes, hipStream_t stream);

const char *fastmax_strerror(int code);

/*
 * Segments of the causal MFMA scans (bf16, D = 64, p = 2: the forward and
 * the backward's dv scan).  These scans carry the moment state of Sec. 2.4's
 * causal recurrences (Eqs. "xcausal", "ycausal") across 128-token chunks,
 * one workgroup per (head, 16-column slice).  A split cuts each such scan at
 * a chunk boundary into two workgroups: the first scans its chunks and then
 * emits its summary (the moment sums over its tokens, which are the exclusive
 * prefix of the second), the second starts from that summary.
 *   FASTMAX_SCAN_SEGMENTS_AUTO (default): split the forward's scans when
 *     two half-length workgroups per scan fill the GPU's 256 CUs in fewer
 *     rounds than one (e.g. B*H = 96; not B*H = 64); the backward's dv scan
 *     is not split (it shares its launch with the in-chunk gradient blocks,
 *     which already fill its last round);
 *   FASTMAX_SCAN_SEGMENTS_OFF: never split;
 *   FASTMAX_SCAN_SEGMENTS_ON: split both scans for every sequence of two
 *     chunks or more;
 *   FASTMAX_SCAN_SEGMENTS_REBUILD: as ON, but the second workgroup rebuilds
 *     the first's summary itself (state updates over the earlier chunks)
 *     instead of waiting for it -- the path a second workgroup also takes
 *     if the summary has not arrived within about 0.3 s.
 * Every mode gives bit-identical results; the workspace sizes do not depend
 * on the mode.  The mode is process-wide and applies to calls made after
 * this returns.  Returns the previous mode, or FASTMAX_EINVAL for any other
 * value.
 */
#define FASTMAX_SCAN_SEGMENTS_AUTO 0
#define FASTMAX_SCAN_SEGMENTS_OFF 1
#define FASTMAX_SCAN_SEGMENTS_ON 2
#define FASTMAX_SCAN_SEGMENTS_REBUILD 3
int fastmax_set_scan_segments(int mode);

/* Library version as "major.minor.patch". */
const char *fastmax_version(void);

/*
 * Allocation-free forward, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * it).  Arguments, layouts, results and errors are those of
 * fastmax_fwd_scaled, without the workspace: the library uses a static
 * device array of FASTMAX_NOALLOC_MAX_WORKSPACE_BYTES (64 MiB) per GPU
 * instead, which each GPU the library runs on holds until the process ends.
 * Problems whose fastmax_workspace_bytes(..., backward = 0) exceeds that
 * size are rejected with FASTMAX_EWORKSPACE before anything is enqueued
 * (e.g. the causal bf16, D = 64, p = 2 forward, whose workspace holds q^ and
 * k^ in fp16 and about 0.4 MB of scan-segment summaries per head, takes one
 * head of up to 260594 tokens, or up to 46 heads of 4096 tokens; the D = 128,
 * p = 2 forward keeps four partial float32 numerators per token, about 2 KB
 * per token and head, and takes 8 heads of up to 4064 tokens, or one head of
 * up to 11081).  The call allocates nothing (no hipMalloc, no library
 * allocation);
 * the first call on a GPU looks the array's device address up once
 * (FASTMAX_EHIP if HIP refuses).  The array used is the current device's,
 * which is why the stream must belong to that device (as for every call).  Every call on one GPU shares that GPU's
 * array: calls whose work overlaps on one GPU (different streams without
 * ordering, or several host threads) race on it and must be serialised by
 * the caller.  The array keeps the last call's contents; no forward path
 * needs it zeroed.
 */
#define FASTMAX_NOALLOC_MAX_WORKSPACE_BYTES ((size_t)64 << 20)
int fastmax_fwd_noalloc(const void *q, const void *k, const void *v, void *out,
                        float *g, int B, int H, int N, int D, int p, int causal,
                        float qk_scale, fastmax_dtype_t dt, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* FASTMAX_H */

// Internal launch interface between the C ABI (api.cpp) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace fm {

// The forward behind the C ABI in three steps (api.cpp): host-side argument
// checks (a FASTMAX_* code), the workspace it needs, and the launch on the
// path that serves the configuration (a FASTMAX_* code).  dt is a
// fastmax_dtype_t.
int fwd_validate(const void *q, const void *k, const void *v, const void *out, const float *g,
                 int B, int H, int N, int D, int p, int causal, float qk_scale, int dt);
// A launch of `blocks` workgroups of `threads` work-items along one grid
// dimension fits the dispatch limits: at most 2^31 - 1 workgroups and
// 2^32 - 1 work-items.  Every launcher checks all the grids of a call with it
// before its first launch (hipErrorInvalidConfiguration otherwise).
inline bool grid_fits(long long blocks, long long threads)
{
    return blocks >= 1 && blocks <= 0x7fffffffLL && blocks * threads <= 0xffffffffLL;
}
// The float32 MFMA forward's grids (also those of the backward's dv scan) and
// the segmented non-causal MFMA path's grids fit.
bool f32mfma_fwd_grids_fit(int BH, int N, int D, int p);
bool mfma_nc_grids_fit(int BH, int N);

// FASTMAX_OK if stream is 0 or belongs to the current device, FASTMAX_EINVAL
// if it belongs to another one, FASTMAX_EHIP if HIP cannot tell.
int check_stream(hipStream_t stream);
size_t fwd_workspace(int B, int H, int N, int D, int p, int causal, int dt);
int fwd_run(const void *q, const void *k, const void *v, void *out, float *g, int B, int H, int N,
            int D, int p, int causal, float qk_scale, int dt, void *workspace, hipStream_t stream);

// Generic float32-VALU path: every (D, p, causal, dtype).
// qs: score scale (weights f_p(qs q^.k^)), applied to q^ where it is
// standardised and to dq^ before the standardisation backward.
hipError_t generic_fwd(const void *q, const void *k, const void *v, void *out, float *g, int BH,
                       int N, int D, int p, int causal, int is_bf16, float qs, void *ws,
                       hipStream_t st);
// Forward workspace of the generic path: per-segment moment states when a
// head's sequence is split into segments (few heads), else 0.
size_t generic_fwd_workspace(int BH, int N, int D, int p);
hipError_t generic_bwd(const void *q, const void *k, const void *v, const void *o,
                       const void *dout, const float *g, void *dq, void *dk, void *dv, int BH,
                       int N, int D, int p, int causal, int is_bf16, float qs, void *ws,
                       hipStream_t st);
size_t generic_bwd_workspace(int B, int H, int N, int D, int p);

// Quadratic-term dropout (p = 2) on the generic kernels: bits are the keep
// bits ([BH][N][mask_words(D)] words), inv = 1 / (1 - rate).  Workspaces:
// generic_fwd_dropout_workspace and generic_bwd_workspace with p = 2.
hipError_t generic_fwd_dropout(const void *q, const void *k, const void *v, void *out, float *g,
                               int BH, int N, int D, int causal, int is_bf16, float qs,
                               const uint32_t *bits, float inv, void *ws, hipStream_t st);
hipError_t generic_bwd_dropout(const void *q, const void *k, const void *v, const void *o,
                               const void *dout, const float *g, void *dq, void *dk, void *dv,
                               int BH, int N, int D, int causal, int is_bf16, float qs,
                               const uint32_t *bits, float inv, void *ws, hipStream_t st);
// Dropout forward workspace: the p = 2 segment states and, causal, the masked
// in-chunk weights (64 bytes per token).
size_t generic_fwd_dropout_workspace(int BH, int N, int D, int causal);
// Philox4x32-10 keep bits for BH heads of N tokens; a feature is kept iff its
// generator word is >= thr.
hipError_t dropout_mask(uint32_t *bits, int BH, int N, int D, uint32_t thr, uint64_t seed,
                        hipStream_t st);

// Two-segment split of the MFMA causal scans (forward and the backward's dv
// scan): whether the (head, slice) items of one launch are split, and where.
// mode: FASTMAX_SCAN_SEGMENTS_* (fastmax.h).
struct ScanSplit {
    int split;    // 0 or 1
    int csplit;   // first chunk of the second segment
    int wait;     // the second segment waits for the first's summary
};
// auto_split: whether the automatic mode may split this launch (the
// backward's dv scan shares its launch with the in-chunk gradient blocks,
// which already fill its last round; there a split only adds work).
ScanSplit causal_scan_split(int items, int nch, bool auto_split);
int set_scan_segment_mode(int mode);
// Summaries and flags of a split scan of `items` (head, slice) items of nch
// chunks (reserved whenever nch >= 2, whatever the mode).
size_t causal_scan_seg_workspace(int items, int nch);

// Float32 MFMA kernels (v_mfma_f32_16x16x4_f32): p in {1, 2}, D in {16, 32,
// 64, 128}, float32 or bf16 I/O, causal and non-causal (dispatch sends bf16
// D = 64 p = 2 here only where the fp16 MFMA kernels do not serve it).  The forward's ws holds
// f32mfma_fwd_workspace(BH, N, D, p) bytes (segment sums; at D = 128, p = 2
// the partial numerators and denominators).
bool f32mfma_applies(int D, int p, int is_bf16);
size_t f32mfma_fwd_workspace(int BH, int N, int D, int p);
hipError_t f32mfma_fwd(const void *q, const void *k, const void *v, void *out, float *g, int BH,
                       int N, int D, int p, int causal, int is_bf16, float qs, void *ws,
                       hipStream_t st);
// The backward's dv_n = sum_{i >= n (causal)} f(s_in) dO_i rg_i (rg = 1/G) on
// the forward's kernels; ws as for the forward.
hipError_t f32mfma_dv(const void *q, const void *k, const void *dout, const float *rg, void *dv,
                      int BH, int N, int D, int p, int causal, int is_bf16, float qs, void *ws,
                      hipStream_t st);
// The backward (same cases as the forward): dq, dk, dv.
size_t f32mfma_bwd_workspace(int BH, int N, int D, int p);
hipError_t f32mfma_bwd(const void *q, const void *k, const void *v, const void *o,
                       const void *dout, const float *g, void *dq, void *dk, void *dv, int BH,
                       int N, int D, int p, int causal, int is_bf16, float qs, void *ws,
                       hipStream_t st);

// MFMA causal scan: D = 64, p = 2, bf16 I/O.
// ws holds mfma_causal_fwd_workspace(BH, N) bytes: q^ and k^ in fp16, then
// the segment summaries and flags.
hipError_t mfma_causal_fwd(const void *q, const void *k, const void *v, void *out, float *g,
                           int BH, int N, float qs, void *ws, hipStream_t st);
size_t mfma_causal_fwd_workspace(int BH, int N);
size_t mfma_causal_smem_bytes();

// MFMA causal backward: D = 64, p = 2, bf16 I/O.  ws holds
// mfma_causal_bwd_workspace(BH, N) bytes.
hipError_t mfma_causal_bwd(const void *q, const void *k, const void *v, const void *o,
                           const void *dout, const float *g, void *dq, void *dk, void *dv, int BH,
                           int N, float qs, void *ws, hipStream_t st);
size_t mfma_causal_bwd_workspace(int BH, int N);

// MFMA non-causal backward: D = 64, p = 2, bf16 I/O, N >= 128 (dv on the
// non-causal forward kernels, dq^ and dk^ by the moment-gradient scans
// against the totals).  ws holds mfma_nc_bwd_workspace(BH, N) bytes.
hipError_t mfma_nc_bwd(const void *q, const void *k, const void *v, const void *o,
                       const void *dout, const float *g, void *dq, void *dk, void *dv, int BH,
                       int N, float qs, void *ws, hipStream_t st);
size_t mfma_nc_bwd_workspace(int BH, int N);

// MFMA non-causal path: D = 64, p = 2, bf16 I/O (moment build, segment
// reduction, query contraction).  ws holds mfma_nc_workspace(BH, N) bytes.
hipError_t mfma_nc_fwd(const void *q, const void *k, const void *v, void *out, float *g, int BH,
                       int N, float qs, void *ws, hipStream_t st);
size_t mfma_nc_workspace(int BH, int N);
// The non-causal backward's dv on the same kernels (keys q^, queries k^, both
// standardised in fp16; values dO scaled per row by rg = 1/G; no divide).
// ws holds mfma_nc_workspace(BH, N) bytes.
hipError_t mfma_nc_dv(const void *qh, const void *kh, const void *dout, const float *rg, void *dv,
                      int BH, int N, void *ws, hipStream_t st);

}  // namespace fm

// C ABI of the Fastmax library: host-side validation, workspace sizing and
// dispatch to the HIP kernels.  Every check runs before anything is enqueued
// (the stream's device is the only one that asks HIP).
#include <stdint.h>
#include <string.h>

#include "../../include/fastmax.h"
#include "fm_common.h"
#include "fm_internal.h"

namespace {

// Head sizes served: 16, 32, 64 and 128 (the last the head size of Sec. 3.1's
// Llama-2 remark).  bf16 D = 64, p = 2 runs on the fp16 MFMA kernels where they
// apply, every other plain call on the float32 MFMA kernels, the dropout
// calls on the generic float32 kernels.
bool supported_d(int D) { return D == 16 || D == 32 || D == 64 || D == 128; }

int check_common(int B, int H, int N, int D, int p, int causal, int dt)
{
    if (B < 1 || H < 1 || N < 1) return FASTMAX_EINVAL;
    if (p != 1 && p != 2) return FASTMAX_EINVAL;
    if (causal != 0 && causal != 1) return FASTMAX_EINVAL;
    if (dt != FASTMAX_F32 && dt != FASTMAX_BF16) return FASTMAX_EINVAL;
    if (!supported_d(D)) return FASTMAX_EUNSUPPORTED;
    // Size limits: B*H*N*D < 2^62; at most 2^20 heads (B*H) and 2^30 tokens
    // per head, so that every chunk, workgroup and row count the launchers
    // derive from them stays within int.
    unsigned __int128 tot = (unsigned __int128)B * H * N * D;
    if (tot >= ((unsigned __int128)1 << 62)) return FASTMAX_EINVAL;
    if ((long long)B * H > (1LL << 20) || N > (1 << 30)) return FASTMAX_EINVAL;
    return FASTMAX_OK;
}

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

// The dtype argument as an int, read without loading it as an enum: a C
// caller may pass any int, and a C++ enum value outside the enumerators'
// range is undefined behaviour (UBSan reports it), so validation reads the
// bits.
int dt_bits(const fastmax_dtype_t *dt)
{
    int v;
    memcpy(&v, dt, sizeof v);
    return v;
}

// The score scale multiplies q^.k^ inside f_p.  (0, 1] covers the definition
// (1) and the unit-norm and temperature variants (1/D, 1/sqrt(D)); the fp16
// moment scaling of the MFMA backward assumes |qs q^_m qs q^_l| <= 64.  NaN
// fails both comparisons.
bool valid_scale(float qs) { return qs > 0.0f && qs <= 1.0f; }

// The segmented MFMA path rounds the moments to fp16; with very few keys G
// can be far smaller than the moment terms it is summed from (G = f_2(s) >= 1/2
// for one key against terms of size ~|q^||k^|^2/2), which amplifies that
// rounding past the bf16 tolerance.  Below one 128-token chunk of keys the
// float32 MFMA kernels take the call: exact to fp32, next to no cost.
bool mfma_noncausal(int N, int D, int p, int causal, int dt)
{
    return D == 64 && p == 2 && !causal && dt == FASTMAX_BF16 && N >= 128;
}

// Drop probability of the quadratic-term dropout: [0, 1) (NaN fails).
bool valid_rate(float rate) { return rate >= 0.0f && rate < 1.0f; }

bool aligned4(const void *p) { return ((uintptr_t)p & 3u) == 0; }

bool mfma_causal(int D, int p, int causal, int dt)
{
    return D == 64 && p == 2 && causal && dt == FASTMAX_BF16;
}

// The float32 MFMA kernels (forward and backward) serve every case the fp16
// MFMA kernels do not (p = 1; p = 2 with float32 I/O, with D != 64, or
// non-causal below 128 tokens).
bool f32mfma(int D, int p, int causal, int dt, int N)
{
    if (mfma_causal(D, p, causal, dt) || mfma_noncausal(N, D, p, causal, dt)) return false;
    return fm::f32mfma_applies(D, p, dt == FASTMAX_BF16);
}

size_t fwd_ws(int B, int H, int N, int D, int p, int causal, int dt)
{
    if (mfma_causal(D, p, causal, dt)) return fm::mfma_causal_fwd_workspace(B * H, N);
    if (mfma_noncausal(N, D, p, causal, dt)) return fm::mfma_nc_workspace(B * H, N);
    if (f32mfma(D, p, causal, dt, N)) return fm::f32mfma_fwd_workspace(B * H, N, D, p);
    return fm::generic_fwd_workspace(B * H, N, D, p);
}

size_t bwd_ws(int B, int H, int N, int D, int p, int causal, int dt)
{
    if (mfma_causal(D, p, causal, dt)) return fm::mfma_causal_bwd_workspace(B * H, N);
    if (mfma_noncausal(N, D, p, causal, dt)) return fm::mfma_nc_bwd_workspace(B * H, N);
    if (f32mfma(D, p, causal, dt, N)) return fm::f32mfma_bwd_workspace(B * H, N, D, p);
    return fm::generic_bwd_workspace(B, H, N, D, p);
}

}  // namespace

namespace fm {

// A launcher's result as a FASTMAX code: hipErrorInvalidConfiguration is
// what the launchers return, before their first launch, for a call whose
// grids exceed the dispatch limits (an unsupported size); anything else from
// HIP is FASTMAX_EHIP.
int code_of(hipError_t e)
{
    if (e == hipSuccess) return FASTMAX_OK;
    return e == hipErrorInvalidConfiguration ? FASTMAX_EUNSUPPORTED : FASTMAX_EHIP;
}

// Kernels run on the current device.  A stream of another device would run
// them there with this device's launch settings (and, for the allocation-free
// forward, this device's scratch array), so such a stream is refused.  The
// null stream is the current device's.
int check_stream(hipStream_t stream)
{
    if (!stream) return FASTMAX_OK;
    int cur = -1;
    hipDevice_t sd = -1;
    if (hipGetDevice(&cur) != hipSuccess || hipStreamGetDevice(stream, &sd) != hipSuccess)
        return FASTMAX_EHIP;
    return sd == cur ? FASTMAX_OK : FASTMAX_EINVAL;
}

int fwd_validate(const void *q, const void *k, const void *v, const void *out, const float *g,
                 int B, int H, int N, int D, int p, int causal, float qk_scale, int dt)
{
    int rc = check_common(B, H, N, D, p, causal, dt);
    if (rc != FASTMAX_OK) return rc;
    if (!valid_scale(qk_scale)) return FASTMAX_EINVAL;
    if (!q || !k || !v || !out) return FASTMAX_ENULL;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out) ||
        (g && !aligned16(g)))
        return FASTMAX_EALIGN;
    return FASTMAX_OK;
}

size_t fwd_workspace(int B, int H, int N, int D, int p, int causal, int dt)
{
    return fwd_ws(B, H, N, D, p, causal, dt);
}

int fwd_run(const void *q, const void *k, const void *v, void *out, float *g, int B, int H, int N,
            int D, int p, int causal, float qk_scale, int dt, void *workspace, hipStream_t stream)
{
    hipError_t e;
    if (mfma_causal(D, p, causal, dt))
        e = mfma_causal_fwd(q, k, v, out, g, B * H, N, qk_scale, workspace, stream);
    else if (mfma_noncausal(N, D, p, causal, dt))
        e = mfma_nc_fwd(q, k, v, out, g, B * H, N, qk_scale, workspace, stream);
    else if (f32mfma(D, p, causal, dt, N))
        e = f32mfma_fwd(q, k, v, out, g, B * H, N, D, p, causal, dt == FASTMAX_BF16, qk_scale,
                        workspace, stream);
    else
        e = generic_fwd(q, k, v, out, g, B * H, N, D, p, causal, dt == FASTMAX_BF16, qk_scale,
                        workspace, stream);
    return fm::code_of(e);
}

}  // namespace fm

namespace {

int fwd_impl(const void *q, const void *k, const void *v, void *out, float *g, int B, int H,
             int N, int D, int p, int causal, float qk_scale, int dt, void *workspace,
             size_t workspace_bytes, hipStream_t stream)
{
    int rc = fm::fwd_validate(q, k, v, out, g, B, H, N, D, p, causal, qk_scale, dt);
    if (rc != FASTMAX_OK) return rc;
    size_t need = fwd_ws(B, H, N, D, p, causal, dt);
    if (need > 0 && (!workspace || workspace_bytes < need)) return FASTMAX_EWORKSPACE;
    if (workspace && !aligned16(workspace)) return FASTMAX_EALIGN;
    if ((rc = fm::check_stream(stream)) != FASTMAX_OK) return rc;
    return fm::fwd_run(q, k, v, out, g, B, H, N, D, p, causal, qk_scale, dt, workspace, stream);
}

int bwd_impl(const void *q, const void *k, const void *v, const void *out, const void *dout,
             const float *g, void *dq, void *dk, void *dv, int B, int H, int N, int D, int p,
             int causal, float qk_scale, int dt, void *workspace, size_t workspace_bytes,
             hipStream_t stream)
{
    int rc = check_common(B, H, N, D, p, causal, dt);
    if (rc != FASTMAX_OK) return rc;
    if (!valid_scale(qk_scale)) return FASTMAX_EINVAL;
    if (!q || !k || !v || !out || !dout || !g || !dq || !dk || !dv) return FASTMAX_ENULL;
    const void *ptrs[] = {q, k, v, out, dout, g, dq, dk, dv};
    for (const void *ptr : ptrs)
        if (!aligned16(ptr)) return FASTMAX_EALIGN;
    size_t need = bwd_ws(B, H, N, D, p, causal, dt);
    if (need > 0 && (!workspace || workspace_bytes < need)) return FASTMAX_EWORKSPACE;
    if (workspace && !aligned16(workspace)) return FASTMAX_EALIGN;
    if ((rc = fm::check_stream(stream)) != FASTMAX_OK) return rc;
    hipError_t e;
    if (mfma_causal(D, p, causal, dt))
        e = fm::mfma_causal_bwd(q, k, v, out, dout, g, dq, dk, dv, B * H, N, qk_scale, workspace,
                                stream);
    else if (mfma_noncausal(N, D, p, causal, dt))
        e = fm::mfma_nc_bwd(q, k, v, out, dout, g, dq, dk, dv, B * H, N, qk_scale, workspace,
                            stream);
    else if (f32mfma(D, p, causal, dt, N))
        e = fm::f32mfma_bwd(q, k, v, out, dout, g, dq, dk, dv, B * H, N, D, p, causal,
                            dt == FASTMAX_BF16, qk_scale, workspace, stream);
    else
        e = fm::generic_bwd(q, k, v, out, dout, g, dq, dk, dv, B * H, N, D, p, causal,
                            dt == FASTMAX_BF16, qk_scale, workspace, stream);
    return fm::code_of(e);
}

}  // namespace

extern "C" {

size_t fastmax_workspace_bytes(int B, int H, int N, int D, int p, int causal,
                               fastmax_dtype_t dt, int backward)
{
    const int d = dt_bits(&dt);
    if (check_common(B, H, N, D, p, causal, d) != FASTMAX_OK) return 0;
    return backward ? bwd_ws(B, H, N, D, p, causal, d) : fwd_ws(B, H, N, D, p, causal, d);
}

int fastmax_fwd_scaled(const void *q, const void *k, const void *v, void *out, float *g, int B,
                       int H, int N, int D, int p, int causal, float qk_scale,
                       fastmax_dtype_t dt, void *workspace, size_t workspace_bytes,
                       hipStream_t stream)
{
    return fwd_impl(q, k, v, out, g, B, H, N, D, p, causal, qk_scale, dt_bits(&dt), workspace,
                    workspace_bytes, stream);
}

int fastmax_fwd(const void *q, const void *k, const void *v, void *out, float *g, int B, int H,
                int N, int D, int p, int causal, fastmax_dtype_t dt, void *workspace,
                size_t workspace_bytes, hipStream_t stream)
{
    return fwd_impl(q, k, v, out, g, B, H, N, D, p, causal, 1.0f, dt_bits(&dt), workspace,
                    workspace_bytes, stream);
}

int fastmax_bwd_scaled(const void *q, const void *k, const void *v, const void *out,
                       const void *dout, const float *g, void *dq, void *dk, void *dv, int B,
                       int H, int N, int D, int p, int causal, float qk_scale,
                       fastmax_dtype_t dt, void *workspace, size_t workspace_bytes,
                       hipStream_t stream)
{
    return bwd_impl(q, k, v, out, dout, g, dq, dk, dv, B, H, N, D, p, causal, qk_scale,
                    dt_bits(&dt), workspace, workspace_bytes, stream);
}

int fastmax_bwd(const void *q, const void *k, const void *v, const void *out, const void *dout,
                const float *g, void *dq, void *dk, void *dv, int B, int H, int N, int D, int p,
                int causal, fastmax_dtype_t dt, void *workspace, size_t workspace_bytes,
                hipStream_t stream)
{
    return bwd_impl(q, k, v, out, dout, g, dq, dk, dv, B, H, N, D, p, causal, 1.0f,
                    dt_bits(&dt), workspace, workspace_bytes, stream);
}

size_t fastmax_dropout_mask_words(int D)
{
    return supported_d(D) ? (size_t)fm::mask_words(D) : 0;
}

int fastmax_dropout_mask(uint32_t *keep_bits, int B, int H, int N, int D, float rate,
                         uint64_t seed, hipStream_t stream)
{
    int rc = check_common(B, H, N, D, 2, 0, FASTMAX_F32);
    if (rc != FASTMAX_OK) return rc;
    if (!valid_rate(rate)) return FASTMAX_EINVAL;
    if (!keep_bits) return FASTMAX_ENULL;
    if (!aligned4(keep_bits)) return FASTMAX_EALIGN;
    if ((rc = fm::check_stream(stream)) != FASTMAX_OK) return rc;
    // floor(rate 2^32) in double: exact for every float rate in [0, 1)
    const uint32_t thr = (uint32_t)((double)rate * 4294967296.0);
    hipError_t e = fm::dropout_mask(keep_bits, B * H, N, D, thr, seed, stream);
    return fm::code_of(e);
}

size_t fastmax_dropout_workspace_bytes(int B, int H, int N, int D, int causal,
                                       fastmax_dtype_t dt, int backward)
{
    if (check_common(B, H, N, D, 2, causal, dt_bits(&dt)) != FASTMAX_OK) return 0;
    return backward ? fm::generic_bwd_workspace(B, H, N, D, 2)
                    : fm::generic_fwd_dropout_workspace(B * H, N, D, causal);
}

int fastmax_fwd_dropout(const void *q, const void *k, const void *v, void *out, float *g,
                        const uint32_t *keep_bits, float rate, int B, int H, int N, int D,
                        int causal, float qk_scale, fastmax_dtype_t dt_arg, void *workspace,
                        size_t workspace_bytes, hipStream_t stream)
{
    const int dt = dt_bits(&dt_arg);
    int rc = check_common(B, H, N, D, 2, causal, dt);
    if (rc != FASTMAX_OK) return rc;
    if (!valid_scale(qk_scale) || !valid_rate(rate)) return FASTMAX_EINVAL;
    if (!q || !k || !v || !out || !keep_bits) return FASTMAX_ENULL;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out) ||
        (g && !aligned16(g)) || !aligned4(keep_bits))
        return FASTMAX_EALIGN;
    size_t need = fm::generic_fwd_dropout_workspace(B * H, N, D, causal);
    if (need > 0 && (!workspace || workspace_bytes < need)) return FASTMAX_EWORKSPACE;
    if (workspace && !aligned16(workspace)) return FASTMAX_EALIGN;
    if ((rc = fm::check_stream(stream)) != FASTMAX_OK) return rc;
    hipError_t e = fm::generic_fwd_dropout(q, k, v, out, g, B * H, N, D, causal,
                                           dt == FASTMAX_BF16, qk_scale, keep_bits,
                                           1.0f / (1.0f - rate), workspace, stream);
    return fm::code_of(e);
}

int fastmax_bwd_dropout(const void *q, const void *k, const void *v, const void *out,
                        const void *dout, const float *g, const uint32_t *keep_bits, float rate,
                        void *dq, void *dk, void *dv, int B, int H, int N, int D, int causal,
                        float qk_scale, fastmax_dtype_t dt_arg, void *workspace,
                        size_t workspace_bytes, hipStream_t stream)
{
    const int dt = dt_bits(&dt_arg);
    int rc = check_common(B, H, N, D, 2, causal, dt);
    if (rc != FASTMAX_OK) return rc;
    if (!valid_scale(qk_scale) || !valid_rate(rate)) return FASTMAX_EINVAL;
    if (!q || !k || !v || !out || !dout || !g || !keep_bits || !dq || !dk || !dv)
        return FASTMAX_ENULL;
    const void *ptrs[] = {q, k, v, out, dout, g, dq, dk, dv};
    for (const void *ptr : ptrs)
        if (!aligned16(ptr)) return FASTMAX_EALIGN;
    if (!aligned4(keep_bits)) return FASTMAX_EALIGN;
    size_t need = fm::generic_bwd_workspace(B, H, N, D, 2);
    if (!workspace || workspace_bytes < need) return FASTMAX_EWORKSPACE;
    if (!aligned16(workspace)) return FASTMAX_EALIGN;
    if ((rc = fm::check_stream(stream)) != FASTMAX_OK) return rc;
    hipError_t e = fm::generic_bwd_dropout(q, k, v, out, dout, g, dq, dk, dv, B * H, N, D,
                                           causal, dt == FASTMAX_BF16, qk_scale, keep_bits,
                                           1.0f / (1.0f - rate), workspace, stream);
    return fm::code_of(e);
}

int fastmax_set_scan_segments(int mode)
{
    if (mode < FASTMAX_SCAN_SEGMENTS_AUTO || mode > FASTMAX_SCAN_SEGMENTS_REBUILD)
        return FASTMAX_EINVAL;
    return fm::set_scan_segment_mode(mode);
}

const char *fastmax_strerror(int code)
{
    switch (code) {
    case FASTMAX_OK: return "success";
    case FASTMAX_EINVAL: return "invalid argument (p, causal, dtype, B/H/N < 1, B*H > 2^20, N > 2^30, qk_scale not in (0, 1], or dropout rate not in [0, 1))";
    case FASTMAX_EUNSUPPORTED: return "unsupported head dimension (D must be 16, 32, 64 or 128) or a problem whose launch grids exceed the dispatch limits";
    case FASTMAX_ENULL: return "required pointer is NULL";
    case FASTMAX_EALIGN: return "pointer not 16-byte aligned";
    case FASTMAX_EWORKSPACE: return "workspace missing or too small";
    case FASTMAX_EHIP: return "HIP runtime error while enqueuing";
    default: return "unknown error code";
    }
}

const char *fastmax_version(void) { return "0.1.0"; }

}  // extern "C"

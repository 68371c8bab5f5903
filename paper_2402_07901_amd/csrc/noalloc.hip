// Allocation-free forward: fastmax_fwd_scaled with its workspace taken from a
// file-scope device array instead of the caller.  For callers that cannot
// allocate device memory (code under HIP graph capture, tight serving
// loops); the array is per GPU, lives until the process ends, and is shared
// by every call on that GPU.
#include <hip/hip_runtime.h>

#include <string.h>

#include <mutex>

#include "../../include/fastmax.h"
#include "fm_internal.h"

namespace {

static_assert(FASTMAX_NOALLOC_MAX_WORKSPACE_BYTES % 256 == 0, "scratch size");

// Host code must not pass this name to a kernel or a copy: in host code it
// stands for a host-side shadow, not for the device copy.  scratch_ptr()
// returns the device address.
__device__ __align__(256) unsigned char scratch[FASTMAX_NOALLOC_MAX_WORKSPACE_BYTES];

constexpr int MAX_DEVICES = 64;
std::mutex scratch_mu;
void *scratch_dev[MAX_DEVICES] = {};

// Device address of the current device's scratch array, looked up once per
// device (with that device current); nullptr if HIP refuses.
void *scratch_ptr()
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAX_DEVICES) return nullptr;
    std::lock_guard<std::mutex> lock(scratch_mu);
    if (!scratch_dev[dev]) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
        scratch_dev[dev] = p;
    }
    return scratch_dev[dev];
}

}  // namespace

extern "C" int fastmax_fwd_noalloc(const void *q, const void *k, const void *v, void *out,
                                   float *g, int B, int H, int N, int D, int p, int causal,
                                   float qk_scale, fastmax_dtype_t dt, hipStream_t stream)
{
    // the dtype's bits, not a load of the enum (a C caller may pass any int)
    int d;
    memcpy(&d, &dt, sizeof d);
    const int rc = fm::fwd_validate(q, k, v, out, g, B, H, N, D, p, causal, qk_scale, d);
    if (rc != FASTMAX_OK) return rc;
    if (fm::fwd_workspace(B, H, N, D, p, causal, d) > FASTMAX_NOALLOC_MAX_WORKSPACE_BYTES)
        return FASTMAX_EWORKSPACE;
    // the scratch array is the current device's: the work must run there
    const int rs = fm::check_stream(stream);
    if (rs != FASTMAX_OK) return rs;
    // No forward kernel relies on zeroed workspace (every buffer in it is
    // written before it is read), so nothing is cleared.
    void *ws = scratch_ptr();
    if (!ws) return FASTMAX_EHIP;
    return fm::fwd_run(q, k, v, out, g, B, H, N, D, p, causal, qk_scale, d, ws, stream);
}

// Causal Fastmax forward on CDNA4 MFMA, head dimension 64, p = 2, bf16 I/O:
// the launches around the scan of fm_causal_scan.h (its header describes the
// scan), and the standardisation of q and k that precedes it.
#include <hip/hip_runtime.h>

#include <limits.h>

#include <atomic>

#include "fm_causal_scan.h"
#include "fm_common.h"
#include "fm_internal.h"
#include "fm_mfma.h"

namespace fm {
namespace mfma_causal {

using namespace mx;

__global__ __launch_bounds__(NTH, 2) void fwd_causal_kernel(const _Float16 *__restrict__ q,
                                                            const _Float16 *__restrict__ k,
                                                            const bf16_t *__restrict__ v,
                                                            bf16_t *__restrict__ out,
                                                            float *__restrict__ g, int N, int BH,
                                                            SegArgs sa)
{
    extern __shared__ __align__(16) unsigned char smem_raw[];
    Smem &sm = *reinterpret_cast<Smem *>(smem_raw);
    scan_block<false>(sm, q, k, v, out, g, nullptr, N, BH, blockIdx.x, BH * NSL, sa);
}

// q^, k^ (Sec. 2.2, Eqs. 6-7) in fp16 for the scan: an octet of lanes per row,
// 32 rows per workgroup.  q^ is multiplied by the score scale qs, so every
// later step sees the scaled score qs q^.k^.
__global__ __launch_bounds__(256) void standardise_qk(const bf16_t *__restrict__ q,
                                                      const bf16_t *__restrict__ k,
                                                      _Float16 *__restrict__ qh,
                                                      _Float16 *__restrict__ kh, size_t rows,
                                                      float qs, unsigned int *__restrict__ flags,
                                                      int nflags)
{
    // the segment flags of the scan that follows start lowered
    if (blockIdx.x == 0)
        for (int i = threadIdx.x; i < nflags; i += 256) flags[i] = 0u;
    const size_t r = (size_t)blockIdx.x * 32 + (threadIdx.x >> 3);
    const int cg = threadIdx.x & 7;
    const bool valid = r < rows;
    float xq[8] = {}, xk[8] = {};
    if (valid) {
        bf16x8_to_f32(*(const uint4 *)(q + r * D + 8 * cg), xq);
        bf16x8_to_f32(*(const uint4 *)(k + r * D + 8 * cg), xk);
    }
    const h8 hq = standardise8(xq, valid, qs), hk = standardise8(xk, valid);
    if (valid) {
        *(h8 *)(qh + r * D + 8 * cg) = hq;
        *(h8 *)(kh + r * D + 8 * cg) = hk;
    }
}

}  // namespace mfma_causal

namespace {

size_t a256(size_t x) { return (x + 255) & ~(size_t)255; }

// The launches fill this many CUs (one scan workgroup per CU): an MI355X.
constexpr long TARGET_CUS = 256;

std::atomic<int> scan_segment_mode{0};

}  // namespace

int set_scan_segment_mode(int mode)
{
    return scan_segment_mode.exchange(mode);
}

// Auto: split when two segments per item take fewer rounds of half-length
// workgroups than one workgroup per item takes rounds (384 items on 256 CUs:
// 3 half rounds instead of 2 full ones; 256 items: no split).
ScanSplit causal_scan_split(int items, int nch, bool auto_split)
{
    const int mode = scan_segment_mode.load();
    if (nch < 2 || mode == 1 || (mode == 0 && !auto_split)) return ScanSplit{0, 0, 1};
    bool split = true;
    if (mode == 0) {
        const long r1 = (items + TARGET_CUS - 1) / TARGET_CUS;
        const long r2 = (2L * items + TARGET_CUS - 1) / TARGET_CUS;
        split = r2 < 2 * r1;
    }
    if (!split) return ScanSplit{0, 0, 1};
    return ScanSplit{1, nch / 2, mode == 3 ? 0 : 1};
}

size_t causal_scan_seg_workspace(int items, int nch)
{
    if (nch < 2) return 0;
    return a256((size_t)items * mfma_causal::SUM_BYTES) + a256((size_t)items * 4);
}

size_t mfma_causal_fwd_workspace(int BH, int N)
{
    const size_t rows = (size_t)BH * N;
    const int nch = (N + mfma_causal::C - 1) / mfma_causal::C;
    return 2 * a256(rows * mx::D * 2) + causal_scan_seg_workspace(BH * mfma_causal::NSL, nch);
}

size_t mfma_causal_smem_bytes() { return sizeof(mfma_causal::Smem); }

hipError_t mfma_causal_fwd(const void *q, const void *k, const void *v, void *out, float *g,
                           int BH, int N, float qs, void *ws, hipStream_t st)
{
    using namespace mfma_causal;
    static_assert(sizeof(Smem) <= 160 * 1024, "LDS budget");
    static_assert(NHT == 2 * C, "one helper thread per (token pair, v half)");
    const size_t rows = (size_t)BH * N;
    const int items = BH * NSL, nch = (N + C - 1) / C;
    const ScanSplit plan = causal_scan_split(items, nch, true);
    if (!grid_fits((long long)((rows + 31) / 32), 256) ||
        !grid_fits((long long)items * (1 + plan.split), NTH))
        return hipErrorInvalidConfiguration;
    unsigned char *p = (unsigned char *)ws;
    _Float16 *qh = (_Float16 *)p;
    p += a256(rows * D * 2);
    _Float16 *kh = (_Float16 *)p;
    p += a256(rows * D * 2);
    SegArgs sa{nullptr, nullptr, plan.split, plan.csplit, plan.wait};
    if (plan.split) {
        sa.sum = p;
        sa.flags = (unsigned int *)(p + a256((size_t)items * SUM_BYTES));
    }
    hipLaunchKernelGGL(standardise_qk, dim3((unsigned)((rows + 31) / 32)), dim3(256), 0, st,
                       (const bf16_t *)q, (const bf16_t *)k, qh, kh, rows, qs, sa.flags,
                       plan.split ? items : 0);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const size_t smem = sizeof(Smem);
    e = hipFuncSetAttribute((const void *)fwd_causal_kernel,
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(fwd_causal_kernel, dim3(items * (1 + plan.split)), dim3(NTH), smem, st,
                       (const _Float16 *)qh, (const _Float16 *)kh, (const bf16_t *)v,
                       (bf16_t *)out, g, N, BH, sa);
    return hipGetLastError();
}

}  // namespace fm

// Eq. 2 (Sec. II-A) on the GPU, behind nmspmm_confusion: the confusion
// matrix between the N:M output C' of Eq. 1 (with its M/N factor) and the
// dense output C of the same A with the unpruned B,
//   W[i][j] = |C'[i][j] - C[i][j]| / (m*n).
// The operation is elementwise and bound by HBM: two 4-byte reads and one
// 4-byte write per output, in a grid-stride loop of 16-byte accesses when
// the three arrays are 16-byte aligned.  Each output is formed in fp64 (the
// fp32 inputs convert exactly; the difference and the quotient are each
// correctly rounded) and rounded once to fp32.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "nmspmm.h"

namespace nmspmm {
namespace {

constexpr int CF_THREADS = 256;
constexpr int64_t CF_MAX_BLOCKS = 8192;   // 32 workgroups per CU, then grid-stride

__device__ __forceinline__ float confusion_of(float s, float d, double mn)
{
    return (float)(fabs((double)s - (double)d) / mn);
}

// W may be the same array as Cs or Cd: every element is read and then written
// by one thread, and no thread touches another's elements.
template <bool VEC>
__global__ __launch_bounds__(CF_THREADS) void nm_confusion_kernel(const float *Cs, const float *Cd, float *W,
                                                                  int64_t total, double mn)
{
    const int64_t stride = (int64_t)gridDim.x * CF_THREADS;
    const int64_t t = (int64_t)blockIdx.x * CF_THREADS + threadIdx.x;
    if constexpr (VEC) {
        const int64_t count4 = total / 4;
        const float4 *s4 = reinterpret_cast<const float4 *>(Cs);
        const float4 *d4 = reinterpret_cast<const float4 *>(Cd);
        float4 *w4 = reinterpret_cast<float4 *>(W);
        for (int64_t e = t; e < count4; e += stride) {
            const float4 s = s4[e], d = d4[e];
            w4[e] = make_float4(confusion_of(s.x, d.x, mn), confusion_of(s.y, d.y, mn),
                                confusion_of(s.z, d.z, mn), confusion_of(s.w, d.w, mn));
        }
        // the last total % 4 elements, one per thread of the first workgroup
        const int64_t e = 4 * count4 + t;
        if (e < total) W[e] = confusion_of(Cs[e], Cd[e], mn);
    } else {
        for (int64_t e = t; e < total; e += stride) W[e] = confusion_of(Cs[e], Cd[e], mn);
    }
}

bool aligned_to(const void *p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

}  // namespace
}  // namespace nmspmm

using namespace nmspmm;

extern "C" nmspmm_status_t nmspmm_confusion(const float *C_sparse, const float *C_dense, float *W, int64_t m,
                                            int64_t n, hipStream_t stream)
{
    if (m < 0 || n < 0) return NMSPMM_ERR_INVALID_ARG;
    if (m == 0 || n == 0) return NMSPMM_OK;
    if (!C_sparse || !C_dense || !W) return NMSPMM_ERR_INVALID_ARG;
    if (m > INT64_MAX / n) return NMSPMM_ERR_UNSUPPORTED;
    if (!aligned_to(C_sparse, 4) || !aligned_to(C_dense, 4) || !aligned_to(W, 4)) return NMSPMM_ERR_UNSUPPORTED;
    const int64_t total = m * n;
    const double mn = (double)m * (double)n;
    const bool vec = aligned_to(C_sparse, 16) && aligned_to(C_dense, 16) && aligned_to(W, 16);
    const int64_t items = vec ? std::max<int64_t>(total / 4, 1) : total;
    const unsigned blocks = (unsigned)std::min<int64_t>(CF_MAX_BLOCKS, (items + CF_THREADS - 1) / CF_THREADS);
    if (vec)
        hipLaunchKernelGGL(nm_confusion_kernel<true>, dim3(blocks), dim3(CF_THREADS), 0, stream, C_sparse, C_dense,
                           W, total, mn);
    else
        hipLaunchKernelGGL(nm_confusion_kernel<false>, dim3(blocks), dim3(CF_THREADS), 0, stream, C_sparse,
                           C_dense, W, total, mn);
    return hipGetLastError() == hipSuccess ? NMSPMM_OK : NMSPMM_ERR_HIP;
}

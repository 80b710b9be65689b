// Roof micro-benchmarks for the MI355X measurements: the HBM read bandwidth
// and the fp32 matrix-core (MFMA) throughput this chip actually reaches, to
// report beside its published peaks (8 TB/s, 157.3 TFLOP/s fp32).  The paper
// measures its own fp32 peak the same way, at a fixed clock (Sec. IV-E).
// Built into libnm_micro.so, separate from the product library.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "nm_micro.h"

namespace {

constexpr int THREADS = 256;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
constexpr int UNROLL = 4;   // 16-byte loads in flight per thread per trip

// Streaming read: every thread reads 16-byte pieces in a grid-stride loop,
// UNROLL pieces per trip, and folds them into an XOR so that no load can be
// dropped; one store per thread, only if the fold hits a value the caller
// passes (never, for any real data: the store exists to keep the loads).
__global__ __launch_bounds__(THREADS) void nm_micro_read_kernel(const u32x4 *__restrict__ src, int64_t n16,
                                                                uint32_t never, uint32_t *__restrict__ sink)
{
    const int64_t stride = (int64_t)gridDim.x * THREADS;
    int64_t i = (int64_t)blockIdx.x * THREADS + threadIdx.x;
    uint32_t acc = 0;
    for (; i + (UNROLL - 1) * stride < n16; i += UNROLL * stride) {
        u32x4 v[UNROLL];
#pragma unroll
        for (int u = 0; u < UNROLL; ++u) v[u] = __builtin_nontemporal_load(src + i + u * stride);
#pragma unroll
        for (int u = 0; u < UNROLL; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
    for (; i < n16; i += stride) {
        const u32x4 v = src[i];
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    if (acc == never) sink[(int64_t)blockIdx.x * THREADS + threadIdx.x] = acc;
}

// fp32 MFMA throughput: each wave keeps CHAINS independent accumulators of
// v_mfma_f32_32x32x2_f32 (32 x 32 x 2 per instruction, 4096 flops per wave),
// enough to cover the instruction's latency, and runs `iters` rounds.
constexpr int CHAINS = 8;

__global__ __launch_bounds__(THREADS) void nm_micro_mfma_kernel(int iters, float *__restrict__ sink)
{
    typedef float f16v __attribute__((ext_vector_type(16)));
    const float a = 1.0f + 1e-3f * (float)(threadIdx.x & 63);
    const float b = 1.0f - 1e-3f * (float)(threadIdx.x >> 6);
    f16v acc[CHAINS];
#pragma unroll
    for (int c = 0; c < CHAINS; ++c)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[c][e] = 0.f;
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int c = 0; c < CHAINS; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc[c], 0, 0, 0);
    }
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < CHAINS; ++c)
#pragma unroll
        for (int e = 0; e < 16; ++e) s += acc[c][e];
    sink[(int64_t)blockIdx.x * THREADS + threadIdx.x] = s;
}

}  // namespace

extern "C" NM_MICRO_API int nm_micro_hbm_read(const void *buf, int64_t bytes, uint32_t *sink, int blocks, hipStream_t stream)
{
    if (!buf || !sink || bytes < 16 || bytes % 16 != 0 || blocks < 1 || blocks > (1 << 20)) return 1;
    if (reinterpret_cast<uintptr_t>(buf) % 16 != 0) return 1;
    hipLaunchKernelGGL(nm_micro_read_kernel, dim3((unsigned)blocks), dim3(THREADS), 0, stream,
                       static_cast<const u32x4 *>(buf), bytes / 16, 0x9e3779b9u, sink);
    return hipGetLastError() == hipSuccess ? 0 : 2;
}

extern "C" NM_MICRO_API int nm_micro_mfma_f32(float *sink, int iters, int blocks, hipStream_t stream)
{
    if (!sink || iters < 1 || blocks < 1 || blocks > (1 << 20)) return 1;
    hipLaunchKernelGGL(nm_micro_mfma_kernel, dim3((unsigned)blocks), dim3(THREADS), 0, stream, iters, sink);
    return hipGetLastError() == hipSuccess ? 0 : 2;
}

extern "C" NM_MICRO_API double nm_micro_mfma_f32_flops(int iters, int blocks)
{
    return 2.0 * 32 * 32 * 2 * CHAINS * (double)iters * (THREADS / 64) * (double)blocks;
}

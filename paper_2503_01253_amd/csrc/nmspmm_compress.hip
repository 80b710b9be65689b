// Device-side packer behind nmspmm_compress_device: the selection of
// Sec. II-A (N kept row-vectors per window of M k-rows and column block of V
// columns, the offline pre-processing of Sec. III-C.1) done on the GPU, for
// pruning on the fly.  It produces the same bytes as the host packer: the
// score of a row-vector is its squared L2 norm over the block's V columns,
// added left to right in fp64 (fp32 squares are exact in fp64, so the score
// and every tie are reproducible bit for bit); a row-vector is kept when
// fewer than N others have a larger score or an equal score and a smaller
// offset; kept offsets are written in increasing order.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "nmspmm.h"
#include "nmspmm_internal.h"

namespace nmspmm {
namespace {

constexpr int PK_THREADS = 256;   // one thread per (column block, offset); M <= 256

// Workgroup: one window g and `bpw` = 256 / M column blocks; thread t handles
// offset o = t % M of block b = first + t / M.
__global__ __launch_bounds__(PK_THREADS) void nm_compress_kernel(
    const float *__restrict__ B, float *__restrict__ Bc, uint8_t *__restrict__ idx, int64_t n,
    int N, int M, int V, int bpw, int64_t wgs_per_window)
{
    __shared__ double score[PK_THREADS];
    __shared__ int kept[PK_THREADS];

    const int t = threadIdx.x;
    const int64_t g = blockIdx.x / wgs_per_window;
    const int64_t q = n / V;
    const int bl = t / M, o = t % M;
    const int64_t b = (blockIdx.x % wgs_per_window) * bpw + bl;
    const bool active = bl < bpw && b < q;

    const float *row = B + (g * M + o) * n + b * V;
    double s = 0.0;
    if (active)
        for (int c = 0; c < V; ++c) s += (double)row[c] * (double)row[c];
    score[t] = s;
    __syncthreads();

    int keep = 0;
    if (active) {
        int rank = 0;   // row-vectors ahead of this one: larger score, or equal and smaller offset
        for (int o2 = 0; o2 < M; ++o2) {
            const double s2 = score[bl * M + o2];
            rank += (s2 > s) || (s2 == s && o2 < o);
        }
        keep = rank < N;
    }
    kept[t] = keep;
    __syncthreads();

    if (active && keep) {
        int pos = 0;   // kept offsets below this one
        for (int o2 = 0; o2 < o; ++o2) pos += kept[bl * M + o2];
        // exactly N are kept for finite scores; a NaN score (outside the
        // contract) could keep more, so stay inside the window's rows
        if (pos >= N) return;
        const int64_t u = g * N + pos;
        idx[u * q + b] = (uint8_t)o;
        float *dst = Bc + u * n + b * V;
        for (int c = 0; c < V; ++c) dst[c] = row[c];
    }
}

bool aligned4(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 3) == 0; }

}  // namespace
}  // namespace nmspmm

using namespace nmspmm;

extern "C" nmspmm_status_t nmspmm_compress_device(const float *B_dense, int64_t k, int64_t n,
                                                  int N, int M, int V, float *Bc, uint8_t *idx,
                                                  hipStream_t stream)
{
    if (!shape_ok(0, n, k, N, M, V)) return NMSPMM_ERR_INVALID_ARG;
    if (!sizes_fit(1, n, k)) return NMSPMM_ERR_UNSUPPORTED;
    if (k == 0 || n == 0) return NMSPMM_OK;
    if (!B_dense || !Bc || !idx) return NMSPMM_ERR_INVALID_ARG;
    if (!aligned4(B_dense) || !aligned4(Bc)) return NMSPMM_ERR_UNSUPPORTED;
    const int64_t G = k / M, q = n / V;
    const int bpw = PK_THREADS / M;
    const int64_t per_window = (q + bpw - 1) / bpw;
    if (G * per_window > INT32_MAX) return NMSPMM_ERR_UNSUPPORTED;
    hipLaunchKernelGGL(nm_compress_kernel, dim3((unsigned)(G * per_window)), dim3(PK_THREADS), 0,
                       stream, B_dense, Bc, idx, n, N, M, V, bpw, per_window);
    return hipGetLastError() == hipSuccess ? NMSPMM_OK : NMSPMM_ERR_HIP;
}

// Device-side packer behind nmspmm_compress_device: the selection of
// Sec. II-A (N kept row-vectors per window of M k-rows and column block of V
// columns, the offline pre-processing of Sec. III-C.1) done on the GPU, for
// pruning on the fly.  It produces the same bytes as the host packer: the
// score of a row-vector is its squared L2 norm over the block's V columns,
// added left to right in fp64 (fp32 squares are exact in fp64, so the score
// and every tie are reproducible bit for bit); a row-vector is kept when
// fewer than N others have a larger score or an equal score and a smaller
// offset; kept offsets are written in increasing order.
//
// The packer is bound by HBM: it reads B once and writes Bc once.  A
// workgroup stages the M x (bpw * V) tile of one window and bpw column
// blocks in LDS with coalesced loads, scores and ranks its row-vectors there,
// and writes the kept rows of Bc with coalesced stores.  Tiles too large for
// the LDS budget (very wide blocks) take a per-thread kernel that reads each
// row-vector straight from global memory.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "nmspmm.h"
#include "nmspmm_internal.h"

namespace nmspmm {
namespace {

constexpr int PK_THREADS = 256;   // one thread per (column block, offset); M <= 256

// Per-thread packer for tiles past the LDS budget.  Workgroup: one window g
// and `bpw` = 256 / M column blocks; thread t handles offset o = t % M of
// block b = first + t / M.
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

constexpr int PK_LDS = 64 * 1024;   // LDS budget of the tiled packer
constexpr int PK_BATCH = 8;          // staging loads in flight per thread

// LDS layout of the tiled packer for bpw blocks: the tile (row stride
// bpw * V + 1 floats, odd so that threads walking different rows of one
// column hit different banks), then the scores, kept flags and the offset
// kept at each position of each block.
struct PackLds {
    int stride;
    size_t score, kept, sel, bytes;
};

__host__ __device__ inline PackLds pack_lds(int M, int N, int V, int bpw)
{
    PackLds l;
    l.stride = bpw * V + 1;
    l.score = ((size_t)M * l.stride * 4 + 7) / 8 * 8;
    l.kept = l.score + (size_t)M * bpw * 8;
    l.sel = l.kept + (size_t)M * bpw * 4;
    l.bytes = l.sel + (size_t)N * bpw * 4;
    return l;
}

// Workgroup: one window g and up to `bpw` column blocks starting at block
// (blockIdx.x % tiles_per_window) * bpw.
__global__ __launch_bounds__(PK_THREADS) void nm_compress_tile_kernel(
    const float *__restrict__ B, float *__restrict__ Bc, uint8_t *__restrict__ idx, int64_t n,
    int N, int M, int V, int bpw, int64_t tiles_per_window)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const PackLds L = pack_lds(M, N, V, bpw);
    float *tile = reinterpret_cast<float *>(smem);
    double *score = reinterpret_cast<double *>(smem + L.score);
    int *kept = reinterpret_cast<int *>(smem + L.kept);
    int *sel = reinterpret_cast<int *>(smem + L.sel);

    const int t = threadIdx.x;
    const int64_t g = blockIdx.x / tiles_per_window;
    const int64_t q = n / V;
    const int64_t b0 = (blockIdx.x % tiles_per_window) * bpw;
    const int nb = (int)(q - b0 < bpw ? q - b0 : bpw);
    const int cols = nb * V;
    const int64_t c0 = b0 * V;
    const int nrv = M * nb;   // row-vectors of this tile, index bl * M + o

    // stage the tile: consecutive threads on consecutive columns, PK_BATCH
    // loads in flight per thread before their LDS writes
    const float *src = B + g * M * n + c0;
    const int total = M * cols;
    for (int e0 = 0; e0 < total; e0 += PK_THREADS * PK_BATCH) {
        float v[PK_BATCH];
#pragma unroll
        for (int i = 0; i < PK_BATCH; ++i) {
            const int e = e0 + i * PK_THREADS + t;
            const int o = e / cols, c = e - o * cols;
            v[i] = e < total ? src[(int64_t)o * n + c] : 0.f;
        }
#pragma unroll
        for (int i = 0; i < PK_BATCH; ++i) {
            const int e = e0 + i * PK_THREADS + t;
            const int o = e / cols, c = e - o * cols;
            if (e < total) tile[o * L.stride + c] = v[i];
        }
    }
    for (int e = t; e < N * nb; e += PK_THREADS) sel[e] = 0;
    __syncthreads();

    for (int rv = t; rv < nrv; rv += PK_THREADS) {
        const int bl = rv / M, o = rv - bl * M;
        const float *x = tile + o * L.stride + bl * V;
        double s = 0.0;
        for (int c = 0; c < V; ++c) s += (double)x[c] * (double)x[c];
        score[rv] = s;
    }
    __syncthreads();

    for (int rv = t; rv < nrv; rv += PK_THREADS) {
        const int bl = rv / M, o = rv - bl * M;
        const double s = score[rv];
        int rank = 0;   // row-vectors ahead of this one: larger score, or equal and smaller offset
        for (int o2 = 0; o2 < M; ++o2) {
            const double s2 = score[bl * M + o2];
            rank += (s2 > s) || (s2 == s && o2 < o);
        }
        kept[rv] = rank < N;
    }
    __syncthreads();

    for (int rv = t; rv < nrv; rv += PK_THREADS) {
        if (!kept[rv]) continue;
        const int bl = rv / M, o = rv - bl * M;
        int pos = 0;   // kept offsets below this one
        for (int o2 = 0; o2 < o; ++o2) pos += kept[bl * M + o2];
        // exactly N are kept for finite scores; a NaN score (outside the
        // contract) could keep more
        if (pos >= N) continue;
        sel[bl * N + pos] = o;
        idx[(g * N + pos) * q + b0 + bl] = (uint8_t)o;
    }
    __syncthreads();

    // the kept rows: consecutive threads on consecutive columns
    float *dst = Bc + g * N * n + c0;
    for (int e = t; e < N * cols; e += PK_THREADS) {
        const int p = e / cols, c = e - p * cols;
        const int o = min(sel[(c / V) * N + p], M - 1);
        dst[(int64_t)p * n + c] = tile[o * L.stride + c];
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
    // tiled packer: about 256 columns per workgroup, fewer where the tile
    // would pass the LDS budget
    int64_t tb = std::max<int64_t>(1, std::min<int64_t>(PK_THREADS / V, q));
    while (tb > 1 && pack_lds(M, N, V, (int)tb).bytes > PK_LDS) --tb;
    const PackLds lds = pack_lds(M, N, V, (int)tb);
    if (lds.bytes <= PK_LDS) {
        const int64_t tiles = (q + tb - 1) / tb;
        if (G * tiles > INT32_MAX) return NMSPMM_ERR_UNSUPPORTED;
        hipLaunchKernelGGL(nm_compress_tile_kernel, dim3((unsigned)(G * tiles)), dim3(PK_THREADS),
                           lds.bytes, stream, B_dense, Bc, idx, n, N, M, V, (int)tb, tiles);
        return hipGetLastError() == hipSuccess ? NMSPMM_OK : NMSPMM_ERR_HIP;
    }
    const int bpw = PK_THREADS / M;
    const int64_t per_window = (q + bpw - 1) / bpw;
    if (G * per_window > INT32_MAX) return NMSPMM_ERR_UNSUPPORTED;
    hipLaunchKernelGGL(nm_compress_kernel, dim3((unsigned)(G * per_window)), dim3(PK_THREADS), 0,
                       stream, B_dense, Bc, idx, n, N, M, V, bpw, per_window);
    return hipGetLastError() == hipSuccess ? NMSPMM_OK : NMSPMM_ERR_HIP;
}

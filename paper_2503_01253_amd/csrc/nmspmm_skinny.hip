// Streaming kernel for short products (m of a few tens of rows), the
// decode-like regime where C = A * B_pruned is bound by reading Bc once from
// HBM (the high-sparsity, memory-bound case of Sec. III-A).
//
// A workgroup owns SK_ROWS rows x COLS columns of C and one slice of the
// windows of k (split-k across workgroups; the workgroups of one output tile
// add into a zeroed C).  The slice is walked in chunks of at most SK_KC
// columns of A:
//   * the chunk of A (SK_ROWS x SK_KC, row-major, contiguous along k) is
//     staged into LDS once, double-buffered, so that the gather of Eq. 1 reads
//     LDS instead of scattering over L2 (the A_s tile of Sec. III-C);
//   * its compressed rows are shared out to the NW waves in runs of QPW quads
//     (4 compressed rows, the MFMA K).  A wave issues its Bc loads straight
//     into MFMA operand registers (BV consecutive columns per lane), then the
//     offset bytes of D for its rows and column blocks, then gathers A from
//     LDS with those offsets and accumulates with v_mfma_f32_16x16x4_f32.
// Bc is read exactly once; no LDS staging is needed for it.  At the end the
// waves' partial tiles are summed through LDS in a fixed order, so one
// workgroup's contribution is deterministic; with split-k the workgroups'
// contributions are added with fp32 atomics.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "nmspmm_skinny.h"
#include "nmspmm_tiled.h"

namespace nmspmm {

namespace {

constexpr int SK_ROWS = 16;     // rows of C per workgroup (one MFMA row tile)
constexpr int SK_NW = 8;        // waves per workgroup
constexpr int SK_NT = SK_NW * 64;
constexpr int SK_KC = 1024;     // columns of A per staged chunk
constexpr int SK_AS = SK_KC + 4;                  // LDS row stride of a staged chunk (floats)
constexpr int SK_ABUF = SK_ROWS * SK_AS;          // floats per chunk buffer
constexpr int SK_A_LD = SK_ROWS * SK_KC / 4 / SK_NT;  // 16-byte A loads per thread and chunk

// Workgroup barrier that waits for this wave's LDS traffic only: global
// loads issued for the next chunk stay in flight across it.
__device__ __forceinline__ void lds_barrier()
{
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(0xF | (7 << 4) | (0 << 8) | (3 << 14));  // lgkmcnt(0)
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

template <int BV, int QPW, int COLS>
__global__ __launch_bounds__(SK_NT) void nm_skinny_kernel(SkinnyArgs p)
{
    constexpr int CG = 16 * BV;             // columns per MFMA column group
    constexpr int NG = COLS / CG;           // column groups per workgroup
    constexpr int RED = SK_NW * SK_ROWS * COLS;
    constexpr int LDS_FLOATS = 2 * SK_ABUF > RED ? 2 * SK_ABUF : RED;
    typedef typename vec_of<BV>::type bvec;

    // two A chunk buffers during the main loop; the reduction area after it
    __shared__ __align__(16) float lds[LDS_FLOATS];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int r = lane & 15, kq = lane >> 4;
    const int tiles_n = p.tiles_n;
    const int tile = blockIdx.x % (p.tiles_m * tiles_n);
    const int split = blockIdx.x / (p.tiles_m * tiles_n);
    const int tm = tile / tiles_n, tn = tile % tiles_n;
    const int64_t row0 = (int64_t)tm * SK_ROWS, col0 = (int64_t)tn * COLS;
    const int64_t m = p.m, n = p.n, k = p.k;
    const int N = p.N, M = p.M, V = p.V;
    const int64_t q = n / V;

    // windows [gb, ge) of this workgroup, walked in chunks of cw windows
    const int64_t G = k / M;
    const int64_t gps = (G + p.splits - 1) / p.splits;
    const int64_t gb = min<int64_t>(G, (int64_t)split * gps), ge = min<int64_t>(G, gb + gps);
    const int cw = p.cw;
    const int64_t nchunks = (ge - gb + cw - 1) / cw;
    // x / N for 0 <= x < 4096 as (x * invN) >> 20 (exact for N <= 256): a
    // chunk holds at most SK_KC / M * N <= 1024 compressed rows
    const uint32_t invN = ((1u << 20) + N - 1) / N;

    const int rows_valid = (int)min<int64_t>(SK_ROWS, m - row0);
    const __amdgpu_buffer_rsrc_t a_rsrc =
        make_rsrc(p.A + row0 * k, (uint32_t)((int64_t)rows_valid * k * 4));

    // ---- A chunk staging: 16-byte loads along k, rows past m read as zero ----
    f32x4 ra[SK_A_LD];
    auto load_a = [&](int64_t c) {
        const int64_t g0 = gb + c * cw;
        const int64_t kc0 = g0 * M, kcn = (min<int64_t>(ge, g0 + cw) - g0) * M;
#pragma unroll
        for (int i = 0; i < SK_A_LD; ++i) {
            const int f = tid + SK_NT * i;
            const int ar = f / (SK_KC / 4), c4 = f % (SK_KC / 4);
            const bool ok = 4 * c4 < kcn;
            const uint32_t off = ok ? (uint32_t)((ar * k + kc0 + 4 * c4) * 4) : OOB;
            // the buffer load returns raw dwords; reinterpret them as floats
            ra[i] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(a_rsrc, (int)off, 0, 0));
        }
    };
    auto store_a = [&](int buf) {
#pragma unroll
        for (int i = 0; i < SK_A_LD; ++i) {
            const int f = tid + SK_NT * i;
            const int ar = f / (SK_KC / 4), c4 = f % (SK_KC / 4);
            *reinterpret_cast<f32x4 *>(lds + buf * SK_ABUF + ar * SK_AS + 4 * c4) = ra[i];
        }
    };

    // column group g of this workgroup: its first column and block
    int64_t gcol[NG];
    int64_t gblk[NG];
#pragma unroll
    for (int g = 0; g < NG; ++g) {
        gcol[g] = col0 + g * CG;
        gblk[g] = gcol[g] / V;
    }

    f32x4 acc[NG][BV];
#pragma unroll
    for (int g = 0; g < NG; ++g)
#pragma unroll
        for (int s = 0; s < BV; ++s) acc[g][s] = f32x4{0.f, 0.f, 0.f, 0.f};

    if (nchunks > 0) {
        load_a(0);
        store_a(0);
    }
    for (int64_t c = 0; c < nchunks; ++c) {
        const int buf = (int)(c & 1);
        if (c + 1 < nchunks) load_a(c + 1);
        // chunk c is in LDS; every wave is done with chunk c-1's buffer
        lds_barrier();
        const int64_t w0 = gb + c * cw;
        const int64_t u0 = w0 * N, u1 = min<int64_t>(ge, w0 + cw) * N;
        const float *As = lds + buf * SK_ABUF + r * SK_AS;
        for (int64_t ub = u0 + (int64_t)wave * QPW * 4; ub < u1; ub += (int64_t)SK_NW * QPW * 4) {
            // 1. Bc, straight into operand registers (independent of D)
            bvec bv[QPW][NG];
#pragma unroll
            for (int j = 0; j < QPW; ++j) {
                const int64_t rows_left = max<int64_t>(0, u1 - (ub + 4 * j));
                const __amdgpu_buffer_rsrc_t b_rsrc =
                    make_rsrc(p.Bc + (ub + 4 * j) * n, (uint32_t)(min<int64_t>(rows_left, 4) * n * 4));
                const bool urow = ub + 4 * j + kq < u1;
#pragma unroll
                for (int g = 0; g < NG; ++g) {
                    const int64_t col = gcol[g] + BV * r;
                    const uint32_t boff = urow && col < n ? (uint32_t)((kq * n + col) * 4) : OOB;
                    // the buffer loads return raw dwords; reinterpret them as floats
                    if constexpr (BV == 4)
                        bv[j][g] = __builtin_bit_cast(
                            f32x4, __builtin_amdgcn_raw_buffer_load_b128(b_rsrc, (int)boff, 0, 0));
                    else if constexpr (BV == 2)
                        bv[j][g] = __builtin_bit_cast(
                            f32x2, __builtin_amdgcn_raw_buffer_load_b64(b_rsrc, (int)boff, 0, 0));
                    else
                        bv[j][g] = __builtin_bit_cast(
                            float, __builtin_amdgcn_raw_buffer_load_b32(b_rsrc, (int)boff, 0, 0));
                }
            }
            // 2. offsets of D for this lane's compressed row and each column block
            int off[QPW][NG];
#pragma unroll
            for (int j = 0; j < QPW; ++j) {
                const int64_t u = ub + 4 * j + kq;
#pragma unroll
                for (int g = 0; g < NG; ++g) {
                    const bool ok = u < u1 && gcol[g] < n;
                    off[j][g] = p.idx[ok ? u * q + gblk[g] : 0];
                }
            }
            // 3. gather A from the staged chunk, MFMAs
#pragma unroll
            for (int j = 0; j < QPW; ++j) {
                const int64_t u = ub + 4 * j + kq;
                const int wbase = u < u1 ? (int)(((uint32_t)(u - u0) * invN) >> 20) * M : 0;
#pragma unroll
                for (int g = 0; g < NG; ++g) {
                    const float a = As[wbase + min(off[j][g], M - 1)];
#pragma unroll
                    for (int s = 0; s < BV; ++s)
                        acc[g][s] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, lane_of<BV>(bv[j][g], s),
                                                                         acc[g][s], 0, 0, 0);
                }
            }
        }
        if (c + 1 < nchunks) store_a(buf ^ 1);
    }

    // ---- sum the waves' partial tiles through LDS (fixed order) ----
    lds_barrier();   // every wave is done reading A chunks
    // lane l holds rows 4*(l/16)+e, columns g*CG + BV*(l%16)+s
    float *mine = lds + wave * SK_ROWS * COLS;
#pragma unroll
    for (int g = 0; g < NG; ++g)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            bvec v;
            if constexpr (BV == 1) {
                v = acc[g][0][e];
            } else {
#pragma unroll
                for (int s = 0; s < BV; ++s) v[s] = acc[g][s][e];
            }
            *reinterpret_cast<bvec *>(mine + (4 * kq + e) * COLS + g * CG + BV * r) = v;
        }
    lds_barrier();
    // one output per lane and step, consecutive lanes on consecutive columns
    // (coalesced stores and atomics)
    constexpr int OUT = SK_ROWS * COLS;
    static_assert(OUT % SK_NT == 0, "reduction split");
#pragma unroll
    for (int e = tid; e < OUT; e += SK_NT) {
        float sum = lds[e];
#pragma unroll
        for (int wv = 1; wv < SK_NW; ++wv) sum += lds[wv * OUT + e];
        const int64_t row = row0 + e / COLS, col = col0 + e % COLS;
        if (row >= m || col >= n) continue;
        if (p.splits == 1)
            p.C[row * n + col] = sum;
        else
            unsafeAtomicAdd(p.C + row * n + col, sum);
    }
}

template <int BV, int QPW, int COLS>
hipError_t launch(const SkinnyArgs &a, hipStream_t stream)
{
    const unsigned grid = (unsigned)a.tiles_m * (unsigned)a.tiles_n * (unsigned)a.splits;
    hipLaunchKernelGGL((nm_skinny_kernel<BV, QPW, COLS>), dim3(grid), dim3(SK_NT), 0, stream, a);
    return hipGetLastError();
}

}  // namespace

int skinny_rows() { return SK_ROWS; }
int skinny_chunk_cols() { return SK_KC; }

// Instantiated (BV, QPW, COLS): the ones that fit in registers without
// spills, with BV * 16 <= COLS.
#define NMSPMM_SKINNY_VARIANTS(X)                                       \
    X(1, 1, 32) X(1, 2, 32) X(1, 4, 32) X(2, 1, 32) X(2, 2, 32) X(2, 4, 32) \
    X(1, 1, 64) X(1, 2, 64) X(2, 1, 64) X(2, 2, 64) X(2, 4, 64)         \
    X(4, 1, 64) X(4, 2, 64) X(4, 4, 64)                                 \
    X(1, 1, 128) X(1, 2, 128) X(2, 1, 128) X(2, 2, 128) X(2, 4, 128)    \
    X(4, 1, 128) X(4, 2, 128) X(4, 4, 128)                              \
    X(1, 1, 256) X(2, 1, 256) X(2, 2, 256) X(4, 1, 256) X(4, 2, 256)

bool skinny_has(int BV, int QPW, int COLS)
{
#define NM_SK_HAS(bv, qpw, cols) \
    if (BV == bv && QPW == qpw && COLS == cols) return true;
    NMSPMM_SKINNY_VARIANTS(NM_SK_HAS)
#undef NM_SK_HAS
    return false;
}

hipError_t launch_skinny(int BV, int QPW, int COLS, const SkinnyArgs &a, hipStream_t stream)
{
#define NM_SK_LAUNCH(bv, qpw, cols) \
    if (BV == bv && QPW == qpw && COLS == cols) return launch<bv, qpw, cols>(a, stream);
    NMSPMM_SKINNY_VARIANTS(NM_SK_LAUNCH)
#undef NM_SK_LAUNCH
    return hipErrorInvalidValue;
}

}  // namespace nmspmm

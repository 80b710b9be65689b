// Streaming kernel for short products (m <= 16 rows of C per workgroup row
// tile), the decode-like regime where C = A * B_pruned is bound by reading
// Bc once from HBM (the high-sparsity, memory-bound case of Sec. III-A).
//
// A workgroup owns SK_ROWS rows x SK_COLS columns of C and one slice of the
// compressed rows (split-k across workgroups; the workgroups of one output
// tile add into a zeroed C).  Its NW waves split that slice again, one run of
// QPW quads (4 compressed rows, the MFMA K) per wave and round:
//   1. every lane loads the offset byte of D for its K row and column group
//      (the index load comes first: the load-load dependency of Sec. III-C.2);
//   2. it then issues, all at once, the loads of its Bc values straight into
//      MFMA operand registers (BV consecutive columns per lane) and its
//      gathered A values (row l%16 of the window column the offset names);
//   3. v_mfma_f32_16x16x4_f32 accumulates.
// No LDS staging is needed on the way in: Bc is read exactly once and A (m x
// k) is small enough to stay in L2.  At the end the waves' partial tiles are
// summed through LDS in a fixed order, so a workgroup's contribution is
// deterministic; with split-k the workgroups' contributions are added with
// fp32 atomics.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "nmspmm_skinny.h"
#include "nmspmm_tiled.h"

namespace nmspmm {

namespace {

constexpr int SK_ROWS = 16;     // rows of C per workgroup (one MFMA row tile)
constexpr int SK_COLS = 256;    // columns of C per workgroup
constexpr int SK_NW = 8;        // waves per workgroup
constexpr int SK_NT = SK_NW * 64;

template <int BV, int QPW>
__global__ __launch_bounds__(SK_NT) void nm_skinny_kernel(SkinnyArgs p)
{
    constexpr int CG = 16 * BV;             // columns per MFMA column group
    constexpr int NG = SK_COLS / CG;        // column groups per workgroup
    typedef typename vec_of<BV>::type bvec;

    __shared__ __align__(16) float red[SK_NW * SK_ROWS * SK_COLS];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int r = lane & 15, kq = lane >> 4;
    const int tiles_n = p.tiles_n;
    const int tile = blockIdx.x % (p.tiles_m * tiles_n);
    const int split = blockIdx.x / (p.tiles_m * tiles_n);
    const int tm = tile / tiles_n, tn = tile % tiles_n;
    const int64_t row0 = (int64_t)tm * SK_ROWS, col0 = (int64_t)tn * SK_COLS;
    const int64_t m = p.m, n = p.n, k = p.k;
    const int N = p.N, M = p.M, V = p.V;
    const int64_t w = (k / M) * N, q = n / V;

    // compressed rows [u_begin, u_end) of this workgroup, whole quads
    const int64_t quads = (w + 3) / 4;
    const int64_t qps = (quads + p.splits - 1) / p.splits;
    const int64_t u_begin = (int64_t)split * qps * 4;
    const int64_t u_end = min<int64_t>(w, u_begin + qps * 4);

    const int rows_valid = (int)min<int64_t>(SK_ROWS, m - row0);
    const __amdgpu_buffer_rsrc_t a_rsrc =
        make_rsrc(p.A + row0 * k, (uint32_t)((int64_t)rows_valid * k * 4));

    // column group g of this workgroup: its first column, block and validity
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

    // rounds: wave wv takes quads wv*QPW .. of each round of NW*QPW quads
    for (int64_t ubase = u_begin; ubase < u_end; ubase += (int64_t)SK_NW * QPW * 4) {
        const int64_t uw = ubase + (int64_t)wave * QPW * 4;   // this wave's first row
        // 1. offsets
        int off[QPW][NG];
#pragma unroll
        for (int j = 0; j < QPW; ++j) {
            const int64_t u = uw + 4 * j + kq;
#pragma unroll
            for (int g = 0; g < NG; ++g) {
                const bool ok = u < u_end && gcol[g] < n;
                off[j][g] = p.idx[ok ? u * q + gblk[g] : 0];
            }
        }
        // 2. Bc (operand layout) and gathered A
        bvec bv[QPW][NG];
        float av[QPW][NG];
#pragma unroll
        for (int j = 0; j < QPW; ++j) {
            const int64_t u = uw + 4 * j + kq;
            const bool urow = u < u_end;
            const int64_t rows_left = max<int64_t>(0, u_end - (uw + 4 * j));
            const __amdgpu_buffer_rsrc_t b_rsrc =
                make_rsrc(p.Bc + (uw + 4 * j) * n, (uint32_t)(min<int64_t>(rows_left, 4) * n * 4));
            const int64_t window = urow ? (u / N) * M : 0;
#pragma unroll
            for (int g = 0; g < NG; ++g) {
                const int64_t col = gcol[g] + BV * r;
                const bool ok = urow && col < n;
                const uint32_t boff = ok ? (uint32_t)((kq * n + col) * 4) : OOB;
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
                const int64_t acol = window + min(off[j][g], M - 1);
                const uint32_t aoff = ok ? (uint32_t)((r * k + acol) * 4) : OOB;
                av[j][g] = __builtin_bit_cast(
                    float, __builtin_amdgcn_raw_buffer_load_b32(a_rsrc, (int)aoff, 0, 0));
            }
        }
        // 3. MFMAs
#pragma unroll
        for (int j = 0; j < QPW; ++j)
#pragma unroll
            for (int g = 0; g < NG; ++g)
#pragma unroll
                for (int s = 0; s < BV; ++s)
                    acc[g][s] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[j][g], lane_of<BV>(bv[j][g], s),
                                                                     acc[g][s], 0, 0, 0);
    }

    // ---- sum the waves' partial tiles through LDS (fixed order) ----
    // lane l holds rows 4*(l/16)+e, columns g*CG + BV*(l%16)+s
    float *mine = red + wave * SK_ROWS * SK_COLS;
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
            *reinterpret_cast<bvec *>(mine + (4 * kq + e) * SK_COLS + g * CG + BV * r) = v;
        }
    __syncthreads();
    constexpr int PER = SK_ROWS * SK_COLS / SK_NT;   // outputs per thread
    static_assert(PER == 8, "reduction split");
#pragma unroll
    for (int h = 0; h < PER / 4; ++h) {
        const int e0 = (tid + h * SK_NT) * 4;         // 4 consecutive outputs
        f32x4 sum = *reinterpret_cast<const f32x4 *>(red + e0);
#pragma unroll
        for (int wv = 1; wv < SK_NW; ++wv)
            sum += *reinterpret_cast<const f32x4 *>(red + wv * SK_ROWS * SK_COLS + e0);
        const int rr = e0 / SK_COLS, cc = e0 % SK_COLS;
        const int64_t row = row0 + rr, col = col0 + cc;
        if (row >= m || col >= n) continue;
        float *dst = p.C + row * n + col;
        if (p.splits == 1) {
            if (col + 3 < n) {
                *reinterpret_cast<f32x4 *>(dst) = sum;
            } else {
                for (int z = 0; z < 4 && col + z < n; ++z) dst[z] = sum[z];
            }
        } else {
            for (int z = 0; z < 4 && col + z < n; ++z) unsafeAtomicAdd(dst + z, sum[z]);
        }
    }
}

template <int BV, int QPW>
hipError_t launch(const SkinnyArgs &a, hipStream_t stream)
{
    const unsigned grid = (unsigned)a.tiles_m * (unsigned)a.tiles_n * (unsigned)a.splits;
    hipLaunchKernelGGL((nm_skinny_kernel<BV, QPW>), dim3(grid), dim3(SK_NT), 0, stream, a);
    return hipGetLastError();
}

}  // namespace

int skinny_rows() { return SK_ROWS; }
int skinny_cols() { return SK_COLS; }

// Instantiated (BV, QPW): every pair that runs without register spills.
bool skinny_has(int BV, int QPW) { return QPW == 1 || QPW == 2 || (QPW == 4 && BV == 4); }

hipError_t launch_skinny(int BV, int QPW, const SkinnyArgs &a, hipStream_t stream)
{
    switch (BV * 16 + QPW) {
    case 4 * 16 + 1: return launch<4, 1>(a, stream);
    case 4 * 16 + 2: return launch<4, 2>(a, stream);
    case 4 * 16 + 4: return launch<4, 4>(a, stream);
    case 2 * 16 + 1: return launch<2, 1>(a, stream);
    case 2 * 16 + 2: return launch<2, 2>(a, stream);
    case 1 * 16 + 1: return launch<1, 1>(a, stream);
    case 1 * 16 + 2: return launch<1, 2>(a, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace nmspmm

// Device half of the C ABI: the gfx950 kernels for vector-wise N:M SpMM and
// the dispatch behind nmspmm_run (Sec. III: tiling, gathered operand fetch,
// double-buffered staging; re-designed for CDNA4 wave64 + fp32 MFMA).
//
// Notation as in the public header: A m x k, Bc w x n, idx w x q (uint8),
// C m x n; w = (k/M)*N, q = n/V; compressed row u belongs to window u/N.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "nmspmm.h"
#include "nmspmm_internal.h"

namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

template <int W> struct vec_of;
template <> struct vec_of<1> { typedef float type; };
template <> struct vec_of<2> { typedef f32x2 type; };
template <> struct vec_of<4> { typedef f32x4 type; };

// ---------------------------------------------------------------------------
// General kernel: any legal (N, M, V) and any alignment.  One thread per
// output column, GEN_ROWS rows per workgroup; every term of Eq. 1 is read
// straight from global memory (the caches serve the reuse).  It exists for
// the shapes the tiled kernel does not cover; it is not tuned.
// ---------------------------------------------------------------------------
constexpr int GEN_COLS = 256;
constexpr int GEN_ROWS = 8;

__global__ __launch_bounds__(GEN_COLS) void nm_general_kernel(
    const float *__restrict__ A, const float *__restrict__ Bc, const uint8_t *__restrict__ idx,
    float *__restrict__ C, int64_t m, int64_t n, int64_t k, int N, int M, int V)
{
    const int64_t j = (int64_t)blockIdx.x * GEN_COLS + threadIdx.x;
    if (j >= n) return;
    const int64_t w = (k / M) * N, q = n / V, b = j / V;
    for (int64_t i0 = (int64_t)blockIdx.y * GEN_ROWS; i0 < m; i0 += (int64_t)gridDim.y * GEN_ROWS) {
        float acc[GEN_ROWS];
#pragma unroll
        for (int r = 0; r < GEN_ROWS; ++r) acc[r] = 0.f;
        for (int64_t u = 0; u < w; ++u) {
            const float bv = Bc[u * n + j];
            const int off = min((int)idx[u * q + b], M - 1);
            const int64_t col = (u / N) * M + off;
#pragma unroll
            for (int r = 0; r < GEN_ROWS; ++r)
                if (i0 + r < m) acc[r] = fmaf(A[(i0 + r) * k + col], bv, acc[r]);
        }
#pragma unroll
        for (int r = 0; r < GEN_ROWS; ++r)
            if (i0 + r < m) C[(i0 + r) * n + j] = acc[r];
    }
}

// ---------------------------------------------------------------------------
// Tiled MFMA kernel.
//
// A workgroup owns a BM x BN tile of C and walks k in stages of KA = 32
// columns of A (KA/M windows, RS = (KA/M)*N compressed rows).  Per stage it
// stages into LDS (Sec. III-B.1, Listing 1's blocking, Sec. III-C.2's double
// buffer):
//   A_s : the whole BM x KA slab of A, stored k-major (A_s[c][i]), so the
//         N:M gather of Eq. 1 becomes "pick LDS row c" and each lane fetches
//         four consecutive output rows with one 16-byte read;
//   B_s : the RS x BN slab of Bc, row-major;
//   X_s : the RS x (BN/V) offsets, pre-converted to byte offsets of A_s rows
//         (the index prefetch of Sec. III-C.2, done once per stage).
// Global loads for stage s+1 are issued into registers before stage s is
// computed and written to the other LDS buffer afterwards: one barrier per
// stage.  The gathered micro-tile contraction (Listing 2's inner kernel) runs
// on v_mfma_f32_16x16x4_f32: fp32 inputs, fp32 accumulation, K = 4
// consecutive compressed rows per instruction, each lane group of 16 taking
// the offset of its own compressed row.
//
// MFMA operand mapping (wave64, 16x16x4): lane l supplies A[l%16][l/16] and
// B[l/16][l%16]; D[4*(l/16)+v][l%16] comes back in element v.  A lanes read
// output rows 4*(l%16)+t of a 64-row chunk (t = 0..3 -> four MFMAs), B lanes
// read columns BV*(l%16)+s of a CG = 16*BV column group that lies inside
// one column block, so all 16 columns of an MFMA share one gather.
// ---------------------------------------------------------------------------
template <int BM_, int BN_, int WM_, int WN_, int BV_>
struct TileCfg {
    static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_, BV = BV_;
    static constexpr int KA = 32;              // A columns per stage
    static constexpr int NW = (BM / WM) * (BN / WN);
    static constexpr int NT = NW * 64;
    static constexpr int AST = BM + 4;         // floats per A_s row (pad: conflict-free writes)
    static constexpr int BST = BN + 4;         // floats per B_s row
    static constexpr int CG = 16 * BV;         // columns per MFMA column group
    static constexpr int NCG = WN / CG;
    static constexpr int NRC = WM / 64;        // 64-row chunks per wave
    static constexpr int A_CHUNKS = (BM / 32) * (KA / 32);
    static constexpr int A_CH_PER_WAVE = A_CHUNKS / NW;
    static constexpr int B_F4_PER_THREAD = (KA * BN / 4 + NT - 1) / NT;
    static constexpr int A_BYTES = KA * AST * 4;
    static_assert(WM % 64 == 0 && WN % CG == 0, "wave tile");
    static_assert(A_CHUNKS % NW == 0, "A chunks must split evenly over waves");
};

// Workgroups are dispatched round-robin over the 8 XCDs.  Renumber them so
// that consecutive logical ids run on one XCD (and share its L2), then walk
// the tiles in groups of GROUP_M tile rows, column-major inside a group, so
// that the workgroups of one XCD share A rows and Bc columns.
__device__ __forceinline__ void map_tile(int pid, int nwg, int tiles_m, int tiles_n, int &tm, int &tn)
{
    constexpr int NXCD = 8, GROUP_M = 4;
    const int xcd = pid % NXCD, local = pid / NXCD;
    const int full = nwg / NXCD, rem = nwg % NXCD;
    const int logical = xcd < rem ? xcd * (full + 1) + local
                                  : rem * (full + 1) + (xcd - rem) * full + local;
    const int per_group = GROUP_M * tiles_n;
    const int group = logical / per_group;
    const int first_m = group * GROUP_M;
    const int gm = min(tiles_m - first_m, GROUP_M);
    const int in_group = logical - group * per_group;
    tm = first_m + in_group % gm;
    tn = in_group / gm;
}

template <class Cfg>
__global__ __launch_bounds__(Cfg::NT) void nm_mfma_kernel(
    const float *__restrict__ A, const float *__restrict__ Bc, const uint8_t *__restrict__ idx,
    float *__restrict__ C, int64_t m, int64_t n, int64_t k, int N, int M, int V,
    int RS, int stages, int tiles_m, int tiles_n, int stage_bytes)
{
    constexpr int BM = Cfg::BM, BN = Cfg::BN, WM = Cfg::WM, WN = Cfg::WN, BV = Cfg::BV;
    constexpr int KA = Cfg::KA, NT = Cfg::NT, AST = Cfg::AST, BST = Cfg::BST;
    constexpr int CG = Cfg::CG, NCG = Cfg::NCG, NRC = Cfg::NRC;
    constexpr int ACH = Cfg::A_CH_PER_WAVE, BF4 = Cfg::B_F4_PER_THREAD;
    typedef typename vec_of<BV>::type bvec;

    extern __shared__ __align__(16) unsigned char lds[];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    int tm, tn;
    map_tile(blockIdx.x, gridDim.x, tiles_m, tiles_n, tm, tn);
    const int64_t row0 = (int64_t)tm * BM, col0 = (int64_t)tn * BN;
    const int64_t w = (int64_t)(k / M) * N, q = n / V;
    const int64_t b_first = col0 / V;
    const int QB = BN >= V ? BN / V : 1;  // column blocks touched by the tile
    const int b_bytes = RS * BST * 4;

    const int wm = wave / (BN / WN), wn = wave % (BN / WN);
    // column block (tile-local) of each of this wave's column groups
    int blk[NCG];
#pragma unroll
    for (int cg = 0; cg < NCG; ++cg)
        blk[cg] = (int)((col0 + wn * WN + cg * CG) / V - b_first);

    // ---- staging registers ----
    f32x4 ra[ACH][4];
    f32x4 rb[BF4];
    int rx = 0;

    auto load_stage = [&](int s) {
        const int64_t kc0 = (int64_t)s * KA;
        const int r8 = lane & 7, c8 = lane >> 3;
#pragma unroll
        for (int ch = 0; ch < ACH; ++ch) {
            const int chunk = wave * ACH + ch;
            const int rbase = (chunk % (BM / 32)) * 32, cbase = (chunk / (BM / 32)) * 32;
            const int64_t kcol = kc0 + cbase + 4 * c8;
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const int64_t row = row0 + rbase + 4 * r8 + t;
                if (row < m && kcol < k)
                    ra[ch][t] = *reinterpret_cast<const f32x4 *>(A + row * k + kcol);
                else
                    ra[ch][t] = f32x4{0.f, 0.f, 0.f, 0.f};
            }
        }
        const int nb4 = RS * (BN / 4);
#pragma unroll
        for (int f = 0; f < BF4; ++f) {
            const int e = tid + f * NT;
            const int ul = e / (BN / 4), c4 = e % (BN / 4);
            const int64_t u = (int64_t)s * RS + ul, col = col0 + 4 * c4;
            if (e < nb4 && u < w && col < n)
                rb[f] = *reinterpret_cast<const f32x4 *>(Bc + u * n + col);
            else
                rb[f] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
        if (tid < RS * QB) {
            const int ul = tid / QB, bl = tid % QB;
            const int64_t u = (int64_t)s * RS + ul, b = b_first + bl;
            int off = 0;
            if (u < w && b < q) off = min((int)idx[u * q + b], M - 1);
            rx = ((ul / N) * M + off) * AST * 4;
        }
    };

    auto store_stage = [&](int p) {
        unsigned char *base = lds + p * stage_bytes;
        float *As = reinterpret_cast<float *>(base);
        float *Bs = reinterpret_cast<float *>(base + Cfg::A_BYTES);
        int *Xs = reinterpret_cast<int *>(base + Cfg::A_BYTES + b_bytes);
        const int r8 = lane & 7, c8 = lane >> 3;
#pragma unroll
        for (int ch = 0; ch < ACH; ++ch) {
            const int chunk = wave * ACH + ch;
            const int rbase = (chunk % (BM / 32)) * 32, cbase = (chunk / (BM / 32)) * 32;
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const f32x4 v = {ra[ch][0][c], ra[ch][1][c], ra[ch][2][c], ra[ch][3][c]};
                *reinterpret_cast<f32x4 *>(As + (cbase + 4 * c8 + c) * AST + rbase + 4 * r8) = v;
            }
        }
        const int nb4 = RS * (BN / 4);
#pragma unroll
        for (int f = 0; f < BF4; ++f) {
            const int e = tid + f * NT;
            if (e < nb4) {
                const int ul = e / (BN / 4), c4 = e % (BN / 4);
                *reinterpret_cast<f32x4 *>(Bs + ul * BST + 4 * c4) = rb[f];
            }
        }
        if (tid < RS * QB) Xs[tid] = rx;
    };

    f32x4 acc[NCG][NRC][4][BV];
#pragma unroll
    for (int cg = 0; cg < NCG; ++cg)
#pragma unroll
        for (int rc = 0; rc < NRC; ++rc)
#pragma unroll
            for (int t = 0; t < 4; ++t)
#pragma unroll
                for (int s = 0; s < BV; ++s) acc[cg][rc][t][s] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int r = lane & 15, kq = lane >> 4;

    auto compute_stage = [&](int p) {
        const unsigned char *base = lds + p * stage_bytes;
        const float *Bs = reinterpret_cast<const float *>(base + Cfg::A_BYTES);
        const int *Xs = reinterpret_cast<const int *>(base + Cfg::A_BYTES + b_bytes);
        const unsigned char *Arow = base + (wm * WM + 4 * r) * 4;
        const float *Bcol = Bs + wn * WN + BV * r;
        for (int quad = 0; quad < RS / 4; ++quad) {
            const int ul = 4 * quad + kq;
            f32x4 a[NCG][NRC];
            bvec b[NCG];
#pragma unroll
            for (int cg = 0; cg < NCG; ++cg) {
                const int xo = Xs[ul * QB + blk[cg]];
#pragma unroll
                for (int rc = 0; rc < NRC; ++rc)
                    a[cg][rc] = *reinterpret_cast<const f32x4 *>(Arow + xo + rc * 64 * 4);
                b[cg] = *reinterpret_cast<const bvec *>(Bcol + ul * BST + cg * CG);
            }
#pragma unroll
            for (int cg = 0; cg < NCG; ++cg)
#pragma unroll
                for (int rc = 0; rc < NRC; ++rc)
#pragma unroll
                    for (int t = 0; t < 4; ++t)
#pragma unroll
                        for (int s = 0; s < BV; ++s) {
                            float bs;
                            if constexpr (BV == 1) bs = b[cg]; else bs = b[cg][s];
                            acc[cg][rc][t][s] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                                a[cg][rc][t], bs, acc[cg][rc][t][s], 0, 0, 0);
                        }
        }
    };

    if (stages > 0) {
        load_stage(0);
        store_stage(0);
    }
    __syncthreads();
    for (int s = 0; s < stages; ++s) {
        const int p = s & 1;
        if (s + 1 < stages) load_stage(s + 1);
        compute_stage(p);
        if (s + 1 < stages) store_stage(p ^ 1);
        __syncthreads();
    }

    // ---- epilogue: lane l holds rows 16*(l/16)+4v+t, columns BV*(l%16)+s ----
#pragma unroll
    for (int cg = 0; cg < NCG; ++cg) {
        const int64_t col = col0 + wn * WN + cg * CG + BV * r;
        if (col >= n) continue;
#pragma unroll
        for (int rc = 0; rc < NRC; ++rc)
#pragma unroll
            for (int v = 0; v < 4; ++v)
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    const int64_t row = row0 + wm * WM + 64 * rc + 16 * kq + 4 * v + t;
                    if (row >= m) continue;
                    bvec out;
                    if constexpr (BV == 1) {
                        out = acc[cg][rc][t][0][v];
                    } else {
#pragma unroll
                        for (int s = 0; s < BV; ++s) out[s] = acc[cg][rc][t][s][v];
                    }
                    *reinterpret_cast<bvec *>(C + row * n + col) = out;
                }
    }
}

// ---------------------------------------------------------------------------
// Dispatch
// ---------------------------------------------------------------------------
enum class Kind { None, General, Large, Small };

using Large1 = TileCfg<256, 256, 128, 64, 1>;
using Large2 = TileCfg<256, 256, 128, 64, 2>;
using Large4 = TileCfg<256, 256, 128, 64, 4>;
using Small1 = TileCfg<128, 128, 64, 64, 1>;
using Small2 = TileCfg<128, 128, 64, 64, 2>;
using Small4 = TileCfg<128, 128, 64, 64, 4>;

struct Plan {
    Kind kind = Kind::None;
    int BV = 0;
    int RS = 0;
};

bool aligned(const void *p, int bytes) { return (reinterpret_cast<uintptr_t>(p) % bytes) == 0; }

Plan make_plan(const float *A, const float *Bc, const float *C, int64_t m, int64_t n, int64_t k,
               int N, int M, int V)
{
    Plan p;
    if (m == 0 || n == 0) return p;
    p.kind = Kind::General;
    // tiled path: windows tile a 32-column stage, 4 | compressed rows per
    // stage (MFMA K), column groups of 16/32/64 inside one column block
    if (!(M == 4 || M == 8 || M == 16 || M == 32)) return p;
    const int RS = (32 / M) * N;
    if (RS % 4 != 0) return p;
    if (V % 16 != 0) return p;
    const int BV = V % 64 == 0 ? 4 : (V % 32 == 0 ? 2 : 1);
    const bool big = m >= 1024 && n >= 1024;
    const int BN = big ? 256 : 128;
    if (!(BN % V == 0 || V % BN == 0)) return p;
    if (!aligned(A, 16) || !aligned(Bc, 16) || !aligned(C, 4 * BV)) return p;
    if (k > INT32_MAX || (n + 256) / 16 > INT32_MAX || (m + 256) / 128 > INT32_MAX) return p;
    p.kind = big ? Kind::Large : Kind::Small;
    p.BV = BV;
    p.RS = RS;
    return p;
}

template <class Cfg>
hipError_t launch_tiled(const float *A, const float *Bc, const uint8_t *idx, float *C, int64_t m,
                        int64_t n, int64_t k, int N, int M, int V, int RS, hipStream_t stream)
{
    const int QB = Cfg::BN >= V ? Cfg::BN / V : 1;
    const int stage_bytes = Cfg::A_BYTES + RS * Cfg::BST * 4 + ((RS * QB * 4 + 15) / 16) * 16;
    const int lds = 2 * stage_bytes;
    const int64_t tiles_m = (m + Cfg::BM - 1) / Cfg::BM, tiles_n = (n + Cfg::BN - 1) / Cfg::BN;
    if (tiles_m * tiles_n > INT32_MAX) return hipErrorInvalidValue;
    const int64_t G = k / M;
    const int gps = Cfg::KA / M;
    const int stages = (int)((G + gps - 1) / gps);
    auto kern = nm_mfma_kernel<Cfg>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, dim3((unsigned)(tiles_m * tiles_n)), dim3(Cfg::NT), lds, stream, A, Bc,
                       idx, C, m, n, k, N, M, V, RS, stages, (int)tiles_m, (int)tiles_n,
                       stage_bytes);
    return hipGetLastError();
}

hipError_t launch_general(const float *A, const float *Bc, const uint8_t *idx, float *C,
                          int64_t m, int64_t n, int64_t k, int N, int M, int V, hipStream_t stream)
{
    const int64_t gx = (n + GEN_COLS - 1) / GEN_COLS;
    const int64_t gy = std::min<int64_t>((m + GEN_ROWS - 1) / GEN_ROWS, 65535);
    if (gx > INT32_MAX) return hipErrorInvalidValue;
    hipLaunchKernelGGL(nm_general_kernel, dim3((unsigned)gx, (unsigned)gy), dim3(GEN_COLS), 0,
                       stream, A, Bc, idx, C, m, n, k, N, M, V);
    return hipGetLastError();
}

}  // namespace

using namespace nmspmm;

extern "C" const char *nmspmm_kernel_name(int64_t m, int64_t n, int64_t k, int N, int M, int V)
{
    if (!shape_ok(m, n, k, N, M, V) || !sizes_fit(m, n, k)) return "invalid";
    // assume well-aligned buffers (what the allocator returns)
    static const float probe[4] = {0, 0, 0, 0};
    const float *al = reinterpret_cast<const float *>(
        (reinterpret_cast<uintptr_t>(probe) + 15) & ~uintptr_t(15));
    const Plan p = make_plan(al, al, al, m, n, k, N, M, V);
    switch (p.kind) {
    case Kind::None: return "none";
    case Kind::General: return "nm_general_kernel";
    case Kind::Large:
        return p.BV == 4 ? "nm_mfma_kernel<256x256,bv4>" : p.BV == 2 ? "nm_mfma_kernel<256x256,bv2>"
                                                               : "nm_mfma_kernel<256x256,bv1>";
    case Kind::Small:
        return p.BV == 4 ? "nm_mfma_kernel<128x128,bv4>" : p.BV == 2 ? "nm_mfma_kernel<128x128,bv2>"
                                                               : "nm_mfma_kernel<128x128,bv1>";
    }
    return "none";
}

extern "C" nmspmm_status_t nmspmm_run(const float *A, const float *Bc, const uint8_t *idx,
                                      float *C, int64_t m, int64_t n, int64_t k, int N, int M,
                                      int V, hipStream_t stream)
{
    if (!shape_ok(m, n, k, N, M, V)) return NMSPMM_ERR_INVALID_ARG;
    if (!sizes_fit(m, n, k)) return NMSPMM_ERR_UNSUPPORTED;
    if (m == 0 || n == 0) return NMSPMM_OK;
    if (!C) return NMSPMM_ERR_INVALID_ARG;
    if (k > 0 && (!A || !Bc || !idx)) return NMSPMM_ERR_INVALID_ARG;
    if (!aligned(C, 4) || (k > 0 && (!aligned(A, 4) || !aligned(Bc, 4))))
        return NMSPMM_ERR_UNSUPPORTED;

    const Plan p = make_plan(A, Bc, C, m, n, k, N, M, V);
    hipError_t e = hipSuccess;
    switch (p.kind) {
    case Kind::None: return NMSPMM_OK;
    case Kind::General: e = launch_general(A, Bc, idx, C, m, n, k, N, M, V, stream); break;
    case Kind::Large:
        e = p.BV == 4 ? launch_tiled<Large4>(A, Bc, idx, C, m, n, k, N, M, V, p.RS, stream)
          : p.BV == 2 ? launch_tiled<Large2>(A, Bc, idx, C, m, n, k, N, M, V, p.RS, stream)
                      : launch_tiled<Large1>(A, Bc, idx, C, m, n, k, N, M, V, p.RS, stream);
        break;
    case Kind::Small:
        e = p.BV == 4 ? launch_tiled<Small4>(A, Bc, idx, C, m, n, k, N, M, V, p.RS, stream)
          : p.BV == 2 ? launch_tiled<Small2>(A, Bc, idx, C, m, n, k, N, M, V, p.RS, stream)
                      : launch_tiled<Small1>(A, Bc, idx, C, m, n, k, N, M, V, p.RS, stream);
        break;
    }
    return e == hipSuccess ? NMSPMM_OK : NMSPMM_ERR_HIP;
}

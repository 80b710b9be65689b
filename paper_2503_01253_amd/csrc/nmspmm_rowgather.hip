// Row-gather kernel for the thinnest products (at most 32 rows of C), in one
// launch with no workspace and no split of k.
//
// Eq. 1 gathers, for compressed row u and column block b, the column
// (u/N)*M + D[u][b] of A.  With at most 32 rows the gathered values of one
// quad (4 consecutive compressed rows, the K of v_mfma_f32_16x16x4_f32) lie in
// at most 32 cache lines of the row-major A, one per row: at M = 32 a window
// of one row is one 128-byte line, and a quad never leaves its window when N
// is a multiple of 4.  Those lines are read straight into MFMA operands from
// L2, where all of A (16 rows x k = 8192: 512 KB) stays while Bc streams past
// it with the non-temporal hint.  Nothing is staged in LDS and nothing is
// transposed first, so the whole product is one launch; each workgroup owns
// a strip of whole columns over all of k, so every output is written once,
// with no zero fill and no atomics.
//
// A workgroup owns all 16*RT rows x one strip of 16*CT columns, inside one
// column block (V a multiple of 16*CT).  Its NW waves split the strip's
// quads and each streams its quads through a ring of D quads in flight in
// registers: per quad a lane loads the D byte of its compressed row (one
// trip ahead), RT floats of A gathered by it, and CT consecutive Bc floats
// (columns CT*(l%16)+s, one per column tile s); it issues RT*CT MFMAs.  The
// waves' partial strips are summed through LDS at the end, in a fixed order.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "nmspmm_rowgather.h"

namespace nmspmm {

namespace {

template <int RT, int CT, int NW>
struct RGShape {
    static constexpr int ROWS = 16 * RT, COLS = 16 * CT;
    static constexpr int RST = COLS + 1;   // LDS row stride of a partial strip
    static constexpr int TILE = ROWS * RST;
    // partial strips held in LDS at once (a power of two dividing NW); the
    // waves beyond them add into the held ones, in wave order
    static constexpr int FIT = (120 * 1024 / 4) / TILE;
    static constexpr int G = FIT >= NW ? NW : FIT >= 8 ? 8 : FIT >= 4 ? 4 : FIT >= 2 ? 2 : 1;
};

template <int CT> struct RGB;
template <> struct RGB<2> { f32x2 v; };
template <> struct RGB<4> { f32x4 v; };

template <int CT, int AUX>
__device__ __forceinline__ void rg_load_b(RGB<CT> &b, __amdgpu_buffer_rsrc_t rs, uint32_t voff, uint32_t soff)
{
    if constexpr (CT == 2)
        b.v = __builtin_bit_cast(f32x2, __builtin_amdgcn_raw_buffer_load_b64(rs, (int)voff, (int)soff, AUX));
    else
        b.v = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, (int)voff, (int)soff, AUX));
}

// AUX: cache policy of the Bc loads (2: non-temporal, the stream leaves L2
// to A).
template <int RT, int CT, int NW, int D, int AUX>
__global__ __launch_bounds__(NW * 64) void nm_rowgather_kernel(const float *__restrict__ A,
                                                              const float *__restrict__ Bc,
                                                              const uint8_t *__restrict__ idx,
                                                              float *__restrict__ C, int m, int64_t n, int k,
                                                              int w, int q, int M, int V, uint32_t magic, uint32_t n1,
                                                              Epilogue epi)
{
    using S = RGShape<RT, CT, NW>;
    constexpr int ROWS = S::ROWS, COLS = S::COLS, RST = S::RST;
    __shared__ float red[S::G * S::TILE];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    // Workgroups are dispatched round-robin over the 8 XCDs: renumber them so
    // that consecutive strips, which gather the same lines of A when they
    // share a column block, run on one XCD and share its L2.
    const int nwg = gridDim.x, pid = blockIdx.x;
    const int xcd = pid % 8, local = pid / 8, full = nwg / 8, rem = nwg % 8;
    const int strip = xcd < rem ? xcd * (full + 1) + local : rem * (full + 1) + (xcd - rem) * full + local;
    const int64_t j0 = (int64_t)strip * COLS;
    const int b = (int)(j0 / V);
    const int nquads = (w + 3) / 4;
    const int qa = (int)((int64_t)wave * nquads / NW);
    const int qb = (int)((int64_t)(wave + 1) * nquads / NW);
    const int nq = qb - qa;

    const int r = lane & 15, kq = lane >> 4;
    // This wave's Bc rows only: quads past its range (the ring loads one trip
    // ahead) read zero and their MFMAs are skipped.  D bytes past w read
    // zero; a compressed row past w gathers nothing (its A offset is out of
    // range and reads zero), so the last partial quad adds zero terms.
    const int u_lo = min(4 * qa, w), u_hi = min(4 * qb, w);
    const auto rs_a = make_rsrc(A, (uint32_t)((int64_t)m * k * 4));
    const auto rs_bc = make_rsrc(Bc + (int64_t)u_lo * n + j0, (uint32_t)((int64_t)(u_hi - u_lo) * n * 4));
    // D bytes come in the aligned dword that holds them (w*q is a multiple
    // of 4, so every such dword lies inside idx); the byte's place in it is
    // the same for all quads of a lane, since a quad spans 4*q bytes
    const auto rs_x = make_rsrc(idx, (uint32_t)((int64_t)w * q));
    const uint32_t lane_bc = (uint32_t)((kq * n + CT * r) * 4);
    const uint32_t quad_bc = (uint32_t)(16 * n);     // bytes of 4 Bc rows
    const uint32_t byte_x = (uint32_t)((int64_t)(4 * qa + kq) * q + b);
    const uint32_t lane_x = byte_x & ~3u, shift_x = 8 * (byte_x & 3u);
    const uint32_t quad_x = (uint32_t)(4 * q);       // D bytes of 4 compressed rows
    // rows past m lie past the end of A and read zero
    const uint32_t lane_a = (uint32_t)(r * k * 4);
    const uint32_t tile_a = (uint32_t)(16 * k * 4);  // bytes of 16 rows of A

    f32x4 acc[RT][CT];
#pragma unroll
    for (int t = 0; t < RT; ++t)
#pragma unroll
        for (int s = 0; s < CT; ++s) acc[t][s] = f32x4{0.f, 0.f, 0.f, 0.f};

    // Ring of D slots: after trip t, slot j holds the operands of quad t*D + j
    // and the D byte of quad (t+1)*D + j.  Trip 0 only loads; every later trip
    // multiplies the previous trip's quads and loads its own.
    float av[D][RT];
    RGB<CT> bv[D];
    uint32_t xv[D];
    // The first trip's D bytes, each slot issued as the loop issues it (A, Bc,
    // D; the A and Bc loads out of range, reading zero), so that the pending
    // loads on entry line up with those of a trip and the wait counts at the
    // loop head stay exact.
#pragma unroll
    for (int j = 0; j < D; ++j) {
#pragma unroll
        for (int t = 0; t < RT; ++t)   // distinct offsets: no two loads merged
            av[j][t] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs_a, (int)(OOB + 1024 * (j * RT + t)), 0, 0));
        rg_load_b<CT, AUX>(bv[j], rs_bc, OOB + 64 * j, 0);
        xv[j] = __builtin_amdgcn_raw_buffer_load_b32(rs_x, (int)lane_x, (int)(j * quad_x), 0);
        __builtin_amdgcn_sched_barrier(0);
    }
    const int trips = (max(nq, 0) + D - 1) / D;
    // one loop, not peeled: a peeled first trip behind its own branch lets
    // the compiler sink its loads, and the wait counts at the loop head
    // become conservative
#pragma clang loop unroll(disable)
    for (int t = 0; t <= trips; ++t) {
#pragma unroll
        for (int j = 0; j < D; ++j) {
            if (t > 0 && (t - 1) * D + j < nq) {
#pragma unroll
                for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                    for (int s = 0; s < CT; ++s)
                        acc[rt][s] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[j][rt], bv[j].v[s], acc[rt][s], 0, 0, 0);
            }
            const int qr = t * D + j;
            // window u/N of the lane's compressed row: magic = ceil(2^32 / N),
            // exact for u < 2^24 (N = 1: magic = 0, n1 = 1)
            const uint32_t u = (uint32_t)(4 * (qa + qr) + kq);
            const uint32_t g = __umulhi(u, magic) + u * n1;
            const uint32_t col = g * (uint32_t)M + min((xv[j] >> shift_x) & 0xffu, (uint32_t)(M - 1));
            const uint32_t aoff = u < (uint32_t)w ? lane_a + 4 * col : OOB;
#pragma unroll
            for (int rt = 0; rt < RT; ++rt)
                av[j][rt] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs_a, (int)(aoff + rt * tile_a), 0, 0));
            rg_load_b<CT, AUX>(bv[j], rs_bc, lane_bc, qr * quad_bc);
            xv[j] = __builtin_amdgcn_raw_buffer_load_b32(rs_x, (int)lane_x, (int)((qr + D) * quad_x), 0);
            // keep each slot's loads right after its MFMAs: gathered to the
            // end of the unrolled body, they would be waited for at once
            __builtin_amdgcn_sched_barrier(0);
        }
    }

    // partial strips of the waves, summed in a fixed order: G held in LDS,
    // the waves beyond them adding into the held ones round by round.  The
    // 16 x 16 MFMA tile holds row 4*(l/16)+e, column l%16 in element e of
    // lane l: row 16*rt + 4*kq + e, column CT*r + s of the strip.
    float *mine = red + (wave % S::G) * S::TILE;
#pragma unroll 1
    for (int round = 0; round < NW / S::G; ++round) {
        if (wave / S::G == round) {
#pragma unroll
            for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                for (int s = 0; s < CT; ++s)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        float &x = mine[(16 * rt + 4 * kq + e) * RST + CT * r + s];
                        x = round == 0 ? acc[rt][s][e] : x + acc[rt][s][e];
                    }
        }
        __syncthreads();
    }
    for (int e = threadIdx.x; e < ROWS * COLS; e += NW * 64) {
        const int row = e / COLS, col = e % COLS;
        float sum = red[row * RST + col];
#pragma unroll
        for (int x = 1; x < S::G; ++x) sum += red[x * S::TILE + row * RST + col];
        if (row < m) C[(int64_t)row * n + j0 + col] = apply_epilogue(epi, sum, j0 + col);
    }
}

template <int RT, int CT, int NW, int D>
hipError_t launch_cfg(const RowGatherArgs &a, hipStream_t stream)
{
    const int w = (int)(a.k / a.M * a.N), q = (int)(a.n / a.V);
    const unsigned strips = (unsigned)(a.n / (16 * CT));
    const uint32_t magic = a.N == 1 ? 0u : (uint32_t)(((uint64_t(1) << 32) + (uint64_t)a.N - 1) / (uint64_t)a.N);
    if (a.stream_b)
        hipLaunchKernelGGL((nm_rowgather_kernel<RT, CT, NW, D, 2>), dim3(strips), dim3(NW * 64), 0, stream, a.A,
                           a.Bc, a.idx, a.C, (int)a.m, a.n, (int)a.k, w, q, a.M, a.V, magic, a.N == 1 ? 1u : 0u, a.epi);
    else
        hipLaunchKernelGGL((nm_rowgather_kernel<RT, CT, NW, D, 0>), dim3(strips), dim3(NW * 64), 0, stream, a.A,
                           a.Bc, a.idx, a.C, (int)a.m, a.n, (int)a.k, w, q, a.M, a.V, magic, a.N == 1 ? 1u : 0u, a.epi);
    return hipGetLastError();
}

// Instantiated configurations: {RT, CT, NW, D}.
#define NM_ROWGATHER_CONFIGS(X)                                                                 \
    X(1, 2, 8, 4) X(1, 2, 8, 8) X(1, 2, 16, 4) X(1, 2, 16, 8)                                   \
    X(1, 4, 8, 4) X(1, 4, 8, 8) X(1, 4, 16, 4) X(1, 4, 16, 8)                                   \
    X(2, 2, 8, 4) X(2, 2, 16, 4) X(2, 4, 8, 4) X(2, 4, 16, 4)

}  // namespace

bool rowgather_has(const RowGatherCfg &c)
{
#define NM_RG_HAS(RT_, CT_, NW_, D_) \
    if (c.RT == RT_ && c.CT == CT_ && c.NW == NW_ && c.D == D_) return true;
    NM_ROWGATHER_CONFIGS(NM_RG_HAS)
#undef NM_RG_HAS
    return false;
}

bool rowgather_fits(const RowGatherCfg &c, int64_t m, int64_t n, int64_t k, int N, int M, int V)
{
    if (!rowgather_has(c) || m > 16 * c.RT || k == 0) return false;
    const int64_t cols = 16 * c.CT;
    if (V % cols != 0) return false;
    const int64_t w = k / M * N, q = n / V, nquads = (w + 3) / 4;
    // the window division (u < 2^24), D read in whole dwords, A offsets of
    // 16*RT rows, Bc and D offsets up to the quads the ring loads past the
    // last one, the grid
    if (w >= (int64_t(1) << 24) || (w * q) % 4 != 0) return false;
    if (16 * c.RT * k * 4 >= (int64_t(1) << 31)) return false;
    if ((4 * nquads + 4 * c.D + 8) * n * 4 >= (int64_t(1) << 31)) return false;
    if ((4 * nquads + 8 * c.D + 8) * q >= (int64_t(1) << 31)) return false;
    return n / cols <= INT32_MAX;
}

hipError_t launch_rowgather(const RowGatherCfg &c, const RowGatherArgs &a, hipStream_t stream)
{
#define NM_RG_LAUNCH(RT_, CT_, NW_, D_) \
    if (c.RT == RT_ && c.CT == CT_ && c.NW == NW_ && c.D == D_) return launch_cfg<RT_, CT_, NW_, D_>(a, stream);
    NM_ROWGATHER_CONFIGS(NM_RG_LAUNCH)
#undef NM_RG_LAUNCH
    return hipErrorInvalidValue;
}

}  // namespace nmspmm

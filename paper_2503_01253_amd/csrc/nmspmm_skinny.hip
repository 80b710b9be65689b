// Streaming kernel for short products (m of a few tens of rows), the
// decode-like regime where C = A * B_pruned is bound by reading Bc once from
// HBM (the high-sparsity, memory-bound case of Sec. III-A).
//
// A workgroup owns SK_ROWS rows x COLS columns of C and one slice of the
// windows of k (split-k across workgroups; the workgroups of one output tile
// add into a zeroed C).  The slice is walked in chunks of at most SK_KC
// columns of A:
//   * each chunk of A (SK_ROWS x SK_KC, row-major) arrives in LDS by
//     buffer->LDS DMA, two chunks in flight in a two-buffer ring, so that
//     the gather of Eq. 1 reads LDS instead of scattering over L2 (the A_s
//     tile of Sec. III-C);
//   * the chunk's compressed rows are shared out to the NW waves in rounds
//     of QPW quads (4 compressed rows, the MFMA K) per wave.  A wave's Bc
//     values go straight from global memory into MFMA operand registers (BV
//     consecutive columns per lane) and its offset bytes of D into
//     registers (the first round's loads are issued before the wait for
//     the chunk's DMA, so the two latencies overlap).  The wave then gathers
//     A from LDS with the offsets and accumulates with
//     v_mfma_f32_16x16x4_f32.
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

constexpr int SK_NW = 8;        // waves per workgroup
constexpr int SK_NT = SK_NW * 64;
constexpr int SK_AREA = 16 * 1024;                // floats of A per chunk (rows x columns)
constexpr int SK_SEG = 256;                       // floats per 16-byte DMA instruction (64 lanes)

// Shape of a workgroup with RT row tiles of 16 rows: its A chunks hold
// SK_AREA / ROWS columns, so that two of them fit in LDS at every RT.
template <int RT>
struct SkShape {
    static constexpr int ROWS = 16 * RT;
    static constexpr int KC = SK_AREA / ROWS;     // columns of A per chunk
    static constexpr int AS = KC + 4;             // LDS row stride of a chunk (floats)
    static constexpr int ABUF = ROWS * AS;        // floats per chunk buffer
    static constexpr int DMA = ROWS * (KC / SK_SEG) / SK_NW;   // DMA instructions per wave and chunk
    static_assert(KC % SK_SEG == 0 && ROWS * (KC / SK_SEG) % SK_NW == 0, "chunk DMA split");
};

// Workgroup barrier after all but the last VM global loads / DMA of this wave
// have completed (vmcnt(VM), VM < 64) and its LDS accesses have too.
template <int VM>
__device__ __forceinline__ void lds_barrier()
{
    static_assert(VM >= 0 && VM < 64, "vmcnt range");
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt((VM & 15) | (7 << 4) | (0 << 8) | ((VM >> 4) << 14));
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// NT: the Bc loads carry the non-temporal hint (cache policy bit 1), for Bc
// much larger than L2: the streamed lines then leave L2 to the A slices, which
// every column tile re-reads.  Measured on MI355X, 16 x 8192 x 8192 at 4:32
// (32 MB of Bc): 15.0 -> 14.4 us; 256 x 256 x 256 at 16:32 (128 KB of Bc,
// which stays in L2 anyway) measured 2 % slower with it.
template <int RT, int BV, int QPW, int COLS, bool NT>
__global__ __launch_bounds__(SK_NT) void nm_skinny_kernel(SkinnyArgs p)
{
    constexpr int BC_AUX = NT ? 2 : 0;
    using SS = SkShape<RT>;
    constexpr int SK_ROWS = SS::ROWS, SK_KC = SS::KC, SK_AS = SS::AS, SK_ABUF = SS::ABUF;
    constexpr int SK_DMA = SS::DMA;
    constexpr int CG = 16 * BV;             // columns per MFMA column group
    constexpr int NG = COLS / CG;           // column groups per workgroup
    // the reduction sums the waves' partial tiles in SLOTS tiles of LDS,
    // SK_NW / SLOTS waves deep
    constexpr int TILE = SK_ROWS * COLS;
    constexpr int LDS_FLOATS = 2 * SK_ABUF > TILE ? 2 * SK_ABUF : TILE;
    constexpr int FIT = LDS_FLOATS / TILE;
    constexpr int SLOTS = FIT >= 8 ? 8 : FIT >= 4 ? 4 : FIT >= 2 ? 2 : 1;
    constexpr int NL = 2 * QPW * NG;        // memory instructions per wave and round
    static_assert(SK_DMA + NL < 64, "vmcnt range");
    static_assert(SK_NW % SLOTS == 0, "reduction passes");
    typedef typename vec_of<BV>::type bvec;

    // two A chunk buffers during the main loop; the reduction area after it
    __shared__ __align__(16) float lds[LDS_FLOATS];

    const int tid = threadIdx.x, lane = tid & 63;
    // uniform across the wave; saying so keeps every address derived from
    // it (the buffer resources included) in scalar registers
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
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
    const int64_t gb = min64(G, (int64_t)split * gps), ge = min64(G, gb + gps);
    const int cw = p.cw;
    const int64_t nchunks = (ge - gb + cw - 1) / cw;
    // x / N for 0 <= x < 4096 as (x * invN) >> 20 (exact for N <= 256): a
    // chunk holds at most SK_KC / M * N <= 1024 compressed rows
    const uint32_t invN = ((1u << 20) + N - 1) / N;

    const int rows_valid = (int)min64(SK_ROWS, m - row0);
    const __amdgpu_buffer_rsrc_t a_rsrc =
        make_rsrc(p.A + row0 * k, (uint32_t)((int64_t)rows_valid * k * 4));

    // ---- A chunk c -> LDS buffer `buf` by DMA; rows past m and columns past
    // the chunk read zero.  Issued unconditionally (valid false: all zeros)
    // so that every wave issues the same memory instructions per chunk. ----
    auto dma_a = [&](int64_t c, int buf, bool valid) {
        const int64_t g0 = gb + c * cw;
        const int64_t kc0 = g0 * M;
        const int64_t kcn = valid ? (min64(ge, g0 + cw) - g0) * M : 0;
#pragma unroll
        for (int i = 0; i < SK_DMA; ++i) {
            const int piece = wave * SK_DMA + i;
            const int ar = piece / (SK_KC / SK_SEG), seg = piece % (SK_KC / SK_SEG);
            const int col = seg * SK_SEG + 4 * lane;
            const uint32_t off = col < kcn ? (uint32_t)((ar * k + kc0 + col) * 4) : OOB;
            lds_dma<16>(a_rsrc, lds + buf * SK_ABUF + ar * SK_AS + seg * SK_SEG, off);
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

    // compressed rows [u0, u1) of chunk c and the first row of this wave's
    // run in round rd
    auto chunk_rows = [&](int64_t c, int64_t &u0, int64_t &u1) {
        const int64_t w0 = gb + c * cw;
        u0 = w0 * N;
        u1 = min64(ge, w0 + cw) * N;
    };

    // Per lane and column group, fixed for the whole kernel: the byte offset
    // of its Bc values and of its offset byte relative to a quad's first
    // compressed row (row kq of the quad).  Bc offsets past the last column
    // get bit 31 (OOB), an offset past every buffer (valid ones stay below
    // 2^31 after the row offset is added: the host keeps 1028 * n * 4 under
    // 2^31).
    uint32_t boff[NG], xoff[NG];
#pragma unroll
    for (int g = 0; g < NG; ++g) {
        const int64_t col = gcol[g] + BV * r;
        boff[g] = (uint32_t)((kq * n + col) * 4) | ((uint32_t)!(col < n) << 31);
        xoff[g] = (uint32_t)(kq * q + gblk[g]);
    }

    // ---- one round's Bc operands and offsets, straight into registers ----
    // One resource per chunk for its Bc rows and one for their offset bytes:
    // rows past the chunk fall outside them and read zero.  (Building the
    // resources per quad kept the scalar unit busier than the matrix pipe.)
    auto load_round = [&](int64_t c, int rd, bvec (&bv)[QPW][NG], int (&off)[QPW][NG]) {
        int64_t u0, u1;
        chunk_rows(c, u0, u1);
        const int64_t nrows = max64(0, u1 - u0);
        const __amdgpu_buffer_rsrc_t b_rsrc = make_rsrc(p.Bc + u0 * n, (uint32_t)(nrows * n * 4));
        const __amdgpu_buffer_rsrc_t x_rsrc = make_rsrc(p.idx + u0 * q, (uint32_t)(nrows * q));
        const uint32_t rb = (uint32_t)((rd * SK_NW + wave) * QPW * 4);   // chunk-relative
#pragma unroll
        for (int j = 0; j < QPW; ++j) {
            const uint32_t rj = rb + 4 * j;                // the quad's first row
            const uint32_t brow = rj * (uint32_t)n * 4, xrow = rj * (uint32_t)q;
#pragma unroll
            for (int g = 0; g < NG; ++g) {
                const int bo = (int)(boff[g] + brow);
                // the buffer loads return raw dwords; reinterpret them as floats
                if constexpr (BV == 4)
                    bv[j][g] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(b_rsrc, bo, 0, BC_AUX));
                else if constexpr (BV == 2)
                    bv[j][g] = __builtin_bit_cast(f32x2, __builtin_amdgcn_raw_buffer_load_b64(b_rsrc, bo, 0, BC_AUX));
                else
                    bv[j][g] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(b_rsrc, bo, 0, BC_AUX));
                off[j][g] = __builtin_amdgcn_raw_buffer_load_b8(x_rsrc, (int)(xoff[g] + xrow), 0, 0);
            }
        }
    };

    f32x4 acc[RT][NG][BV];
#pragma unroll
    for (int t = 0; t < RT; ++t)
#pragma unroll
        for (int g = 0; g < NG; ++g)
#pragma unroll
            for (int s = 0; s < BV; ++s) acc[t][g][s] = f32x4{0.f, 0.f, 0.f, 0.f};

    // ---- gather A from the chunk in `buf`, MFMAs ----
    auto compute = [&](int buf, int64_t u0, int64_t u1, int rd, const bvec (&bv)[QPW][NG],
                       const int (&off)[QPW][NG]) {
        const float *As = lds + buf * SK_ABUF + r * SK_AS;
        // row indices relative to the chunk (fewer than 1024 rows)
        const int nrows = (int)max64(0, u1 - u0);
        const int rb = (rd * SK_NW + wave) * QPW * 4 + kq;
#pragma unroll
        for (int j = 0; j < QPW; ++j) {
            const int ur = rb + 4 * j;
            const int wbase = ur < nrows ? (int)(((uint32_t)ur * invN) >> 20) * M : 0;
#pragma unroll
            for (int g = 0; g < NG; ++g) {
                const int ac = wbase + min(off[j][g], M - 1);
                // one Bc operand feeds the MFMAs of every row tile
#pragma unroll
                for (int t = 0; t < RT; ++t) {
                    const float a = As[t * 16 * SK_AS + ac];
#pragma unroll
                    for (int s = 0; s < BV; ++s)
                        acc[t][g][s] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                            a, lane_of<BV>(bv[j][g], s), acc[t][g][s], 0, 0, 0);
                }
            }
        }
    };

    // ---- chunk loop.  Memory instructions in flight at the barrier that
    // opens chunk c, newest first: the loads of round 0 of chunk c (NL), the
    // DMA of chunk c+1 (SK_DMA); everything older, chunk c's DMA included,
    // must be done.  (Loading the next round, or the next chunk's round,
    // while one is multiplied measured no faster on MI355X.) ----
    bvec bv[QPW][NG];
    int off[QPW][NG];
    if (nchunks > 0) {
        dma_a(0, 0, true);
        dma_a(1, 1, nchunks > 1);
    }
    for (int64_t c = 0; c < nchunks; ++c) {
        int64_t u0, u1;
        chunk_rows(c, u0, u1);
        const int rounds = (int)((u1 - u0 + SK_NW * QPW * 4 - 1) / (SK_NW * QPW * 4));
        load_round(c, 0, bv, off);
        lds_barrier<SK_DMA + NL>();
        for (int rd = 0; rd < rounds; ++rd) {
            if (rd > 0) load_round(c, rd, bv, off);
            compute((int)(c & 1), u0, u1, rd, bv, off);
        }
        // every wave is done with this buffer: refill it with chunk c+2
        lds_barrier<63>();
        dma_a(c + 2, (int)(c & 1), c + 2 < nchunks);
    }
    // no DMA may still be writing LDS when it becomes the reduction area
    lds_barrier<0>();

    // ---- sum the waves' partial tiles through LDS (fixed order) ----
    // lane l holds rows 16*t + 4*(l/16)+e, columns g*CG + BV*(l%16)+s.  In
    // pass i, waves i*SLOTS .. i*SLOTS+SLOTS-1 write (i == 0) or add (i > 0)
    // their tiles into slots 0 .. SLOTS-1.
#pragma unroll
    for (int pass = 0; pass < SK_NW / SLOTS; ++pass) {
        if (wave / SLOTS == pass) {
            float *mine = lds + (wave % SLOTS) * TILE;
#pragma unroll
            for (int t = 0; t < RT; ++t)
#pragma unroll
                for (int g = 0; g < NG; ++g)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        bvec v;
                        if constexpr (BV == 1) {
                            v = acc[t][g][0][e];
                        } else {
#pragma unroll
                            for (int s = 0; s < BV; ++s) v[s] = acc[t][g][s][e];
                        }
                        bvec *dst = reinterpret_cast<bvec *>(mine + (16 * t + 4 * kq + e) * COLS +
                                                             g * CG + BV * r);
                        if (pass == 0) *dst = v;
                        else *dst += v;
                    }
        }
        lds_barrier<0>();
    }
    // one output per lane and step, consecutive lanes on consecutive columns
    // (coalesced stores and atomics)
    static_assert(TILE % SK_NT == 0, "reduction split");
#pragma unroll
    for (int e = tid; e < TILE; e += SK_NT) {
        float sum = lds[e];
#pragma unroll
        for (int sl = 1; sl < SLOTS; ++sl) sum += lds[sl * TILE + e];
        const int64_t row = row0 + e / COLS, col = col0 + e % COLS;
        if (row >= m || col >= n) continue;
        if (p.splits == 1)
            p.C[row * n + col] = apply_epilogue(p.epi, sum, col);
        else
            unsafeAtomicAdd(p.C + row * n + col, sum);
    }
}

template <int RT, int BV, int QPW, int COLS>
hipError_t launch(const SkinnyArgs &a, hipStream_t stream)
{
    const unsigned grid = (unsigned)a.tiles_m * (unsigned)a.tiles_n * (unsigned)a.splits;
    if (a.stream_b)
        hipLaunchKernelGGL((nm_skinny_kernel<RT, BV, QPW, COLS, true>), dim3(grid), dim3(SK_NT), 0, stream, a);
    else
        hipLaunchKernelGGL((nm_skinny_kernel<RT, BV, QPW, COLS, false>), dim3(grid), dim3(SK_NT), 0, stream, a);
    return hipGetLastError();
}

}  // namespace

int skinny_rows(int RT) { return 16 * RT; }
int skinny_chunk_cols(int RT) { return SK_AREA / (16 * RT); }

// Instantiated (RT, BV, QPW, COLS): the ones that fit in registers without
// spills, with BV * 16 <= COLS.
#define NMSPMM_SKINNY_VARIANTS(X)                                                              \
    X(1, 1, 1, 32) X(1, 1, 2, 32) X(1, 1, 4, 32) X(1, 1, 8, 32) X(1, 2, 1, 32) X(1, 2, 2, 32)   \
    X(1, 2, 4, 32) X(1, 2, 8, 32) X(1, 1, 1, 64) X(1, 1, 2, 64) X(1, 1, 4, 64) X(1, 2, 1, 64)   \
    X(1, 2, 2, 64) X(1, 2, 4, 64) X(1, 4, 1, 64) X(1, 4, 2, 64) X(1, 4, 4, 64) X(1, 4, 8, 64)   \
    X(1, 1, 1, 128) X(1, 1, 2, 128) X(1, 2, 1, 128) X(1, 2, 2, 128) X(1, 2, 4, 128)            \
    X(1, 4, 1, 128) X(1, 4, 2, 128) X(1, 4, 4, 128)                                            \
    X(1, 1, 1, 256) X(1, 2, 1, 256) X(1, 2, 2, 256) X(1, 4, 1, 256) X(1, 4, 2, 256)            \
    X(2, 2, 1, 128) X(2, 2, 2, 128) X(2, 4, 1, 128) X(2, 4, 2, 128) X(2, 4, 4, 128)            \
    X(2, 2, 1, 256) X(2, 2, 2, 256) X(2, 4, 1, 256)

bool skinny_has(int RT, int BV, int QPW, int COLS)
{
#define NM_SK_HAS(rt, bv, qpw, cols) \
    if (RT == rt && BV == bv && QPW == qpw && COLS == cols) return true;
    NMSPMM_SKINNY_VARIANTS(NM_SK_HAS)
#undef NM_SK_HAS
    return false;
}

hipError_t launch_skinny(int RT, int BV, int QPW, int COLS, const SkinnyArgs &a, hipStream_t stream)
{
#define NM_SK_LAUNCH(rt, bv, qpw, cols) \
    if (RT == rt && BV == bv && QPW == qpw && COLS == cols) return launch<rt, bv, qpw, cols>(a, stream);
    NMSPMM_SKINNY_VARIANTS(NM_SK_LAUNCH)
#undef NM_SK_LAUNCH
    return hipErrorInvalidValue;
}

}  // namespace nmspmm

// Pipelined streaming kernel for short and medium products (m of tens to a
// few hundred rows), where C = A * B_pruned is bound by moving Bc and the A
// slice into the compute units rather than by the matrix pipe alone.
//
// A workgroup owns ROWS = 16*RT rows x COLS columns of C and one slice of the
// windows of k (split-k across workgroups; the workgroups of one output tile
// add into a zeroed C).  The slice is walked in stages of sw windows: sw*M
// columns of A and sw*N compressed rows of Bc (the k_s x n_s / w_s x n_s
// blocks of Sec. III-B).  Each stage lands in one slot of an NB-slot LDS ring:
//   A_s : ROWS x KS floats of A, row-major, rows padded by 4 floats (the
//         whole slab: the non-packing load of Sec. III-C.1);
//   B_s : RB x COLS floats of Bc, row-major (rows past the stage read zero);
//   X_s : RB x QBMAX offset bytes of D, one zero-extended dword each.
// Two kinds of waves share the workgroup:
//   * NL loader waves issue only buffer -> LDS DMA, NB-1 stages ahead of the
//     compute waves.  A wave issues its memory instructions in order and
//     stalls while the memory pipeline is full; on the loader waves that
//     stall costs nothing, so the matrix pipes are fed while the next stages
//     stream in (the overlap of loads and FMAs of Sec. III-C.2).
//   * NC compute waves touch only LDS.  Compute wave c owns CW = CPW*16*BV
//     consecutive columns of the tile.  For each quad of 4 compressed rows
//     (the K of v_mfma_f32_16x16x4_f32) a lane reads its offset from X_s,
//     gathers A_s[row][window*M + offset] (Eq. 1) for each of its RT row
//     tiles and its BV Bc values from B_s, and accumulates.  Every output
//     belongs to one wave, so no reduction between waves is needed.
// One barrier per stage: before it the loaders wait (vmcnt) until stage s
// has landed; after it they refill the slot that stage s-1 used, which every
// compute wave has finished reading.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "nmspmm_stream.h"

namespace nmspmm {

namespace {

constexpr int PS_NC = 8;                     // compute waves
constexpr int PS_NL = 4;                     // loader waves (one per SIMD)
constexpr int PS_NT = (PS_NC + PS_NL) * 64;
constexpr int PS_KS = 128;                   // columns of A per stage

template <int RT, int BV, int CPW, int RB>
struct PsShape {
    static constexpr int ROWS = 16 * RT;
    static constexpr int CG = 16 * BV;                  // columns per MFMA column group
    static constexpr int CW = CG * CPW;                 // columns per compute wave
    static constexpr int COLS = PS_NC * CW;
    static constexpr int QBMAX = PS_NC * CPW;           // column blocks per tile, at most
    // A_s holds rows in pairs: one 1 KB DMA instruction fills row i and row
    // i + H (H = 16, or 8 with RT = 1; KS = 128 floats each, back to back),
    // and pairs are 4 floats apart.  With RT >= 2 the 16 rows one MFMA
    // gathers (one row of each of 16 pairs) fall in 16 different banks; with
    // RT = 1 they fall in 8, two rows each.
    static_assert(PS_KS == 128, "A_s layout: 32 lanes per row");
    static constexpr int H = RT >= 2 ? 16 : 8;           // row distance inside a pair
    static constexpr int AST = 2 * PS_KS + 4;           // pair stride (floats)
    static constexpr int A_FLOATS = ROWS / 2 * AST;
    // B_s rows are 32 floats (32 banks) longer than a row of the tile, so the
    // two quad rows read by each half of a wave fall in different banks
    static constexpr int BST = COLS + 32;
    static constexpr int B_FLOATS = RB * BST;
    static constexpr int STAGE = A_FLOATS + B_FLOATS;   // floats per ring slot
    // DMA instructions per stage: one per A row pair, 16-byte pieces of up
    // to 64 lanes per Bc row, 64 offset bytes each
    static constexpr int PB = COLS >= 256 ? COLS / 256 : 1;   // pieces per Bc row
    static constexpr int LB = COLS >= 256 ? 64 : COLS / 4;    // lanes per Bc piece
    static constexpr int IA = ROWS / 2, IB = RB * PB, IX = (RB * QBMAX + 63) / 64;
    static constexpr int X_INTS = IX * 64;              // padded: every DMA lane lands inside
    static constexpr int I = IA + IB + IX;
    static constexpr int CMAX = (I + PS_NL - 1) / PS_NL;         // per loader wave, at most
    // ring depth: NB slots of A_s and B_s and NB+1 of X_s (a stage's offsets
    // travel with the previous stage) in LDS, at most NB_MAX, within the range
    // of the loaders' vmcnt (NB-2 stages of CMAX instructions in flight).  A
    // shallow ring measured faster than a deep one: more stages in flight
    // mostly wait in the memory queues (MI355X, graph replay, 4:32:
    // 512 x 512 x 512 6.98 -> 6.43 us at NB_MAX 6 -> 3, 512 x 1024 x 1024
    // 9.60 -> 8.63, 512 x 2048 x 2048 15.72 -> 14.97, 1024 x 2048 x 2048
    // 21.71 -> 21.22; 8:32 and the 8192-wide products unchanged).
    static constexpr int NB_MAX = 3;
    static constexpr int LDS_FLOATS = 160 * 1024 / 4;
    static constexpr int NB_LDS = (LDS_FLOATS - X_INTS) / (STAGE + X_INTS);
    static constexpr int NB_VM = 2 + 63 / CMAX;
    static constexpr int NB = NB_LDS < NB_VM ? (NB_LDS < NB_MAX ? NB_LDS : NB_MAX) : (NB_VM < NB_MAX ? NB_VM : NB_MAX);
    static_assert(NB >= 2, "the schedule keeps at least one stage in flight");
    static constexpr int X_BASE = NB * STAGE;           // X_s ring after the A_s / B_s ring
    static constexpr int TOTAL = NB * STAGE + (NB + 1) * X_INTS;
    // split-k epilogue: the tile, staged row-major for coalesced atomics
    static constexpr int CST = COLS + 4;
    static_assert(LB <= 64 && COLS % 4 == 0, "DMA pieces");
    static_assert(NB >= 2, "LDS ring");
    static_assert(RB % 4 == 0, "stage rows");
    static_assert(ROWS * CST <= TOTAL, "epilogue staging");
    static_assert(IA % PS_NL == 0 && IB % PS_NL == 0, "loader split");
    // A_s offset (floats) of row 16t + r: row 32u + i and row 32u + 16 + i
    // share pair 16u + i (RT >= 2); row i and row i + 8 share pair i (RT = 1)
    __device__ static int a_lane_base(int r) { return RT >= 2 ? r * AST : (r & 7) * AST + (r >> 3) * PS_KS; }
    static constexpr int a_row(int t) { return (t / 2) * 16 * AST + (t & 1) * PS_KS; }
};

// s_waitcnt vmcnt(cnt) lgkmcnt(0) for a wave-uniform cnt in [LO, HI]: a
// tree of scalar branches down to the immediate form.
template <int LO, int HI>
__device__ __forceinline__ void vm_wait_le(int cnt)
{
    if constexpr (LO == HI) {
        static_assert(LO >= 0 && LO < 64, "vmcnt range");
        __builtin_amdgcn_s_waitcnt((LO & 15) | (7 << 4) | (0 << 8) | ((LO >> 4) << 14));
    } else {
        constexpr int MID = (LO + HI) / 2;
        if (cnt <= MID) vm_wait_le<LO, MID>(cnt);
        else vm_wait_le<MID + 1, HI>(cnt);
    }
}

__device__ __forceinline__ void ps_barrier()
{
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// s_waitcnt lgkmcnt(0): this wave's LDS reads have returned
__device__ __forceinline__ void lds_drain()
{
    __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14));
}

// Split-k through a caller-provided workspace:
// workgroup `split` of output tile `tile` stores its partial tile, ROWS x COLS
// floats given by part(e) for e = row * COLS + col, into its own slice of
// `ws` with coalesced stores; a second kernel (nm_splitk_reduce_kernel) sums
// the slices in split order and writes C.  Every thread of the workgroup
// calls this.
template <int ROWS, int COLS, int NT, class Part>
__device__ __forceinline__ void splitk_store(Part part, float *__restrict__ ws, int tile, int split, int splits)
{
    float *mine = ws + ((int64_t)tile * splits + split) * (ROWS * COLS);
    for (int e = threadIdx.x; e < ROWS * COLS; e += NT) mine[e] = part(e);
}

template <int RT, int BV, int CPW, int RB>
__global__ __launch_bounds__(PS_NT) void nm_stream_kernel(StreamArgs p)
{
    using S = PsShape<RT, BV, CPW, RB>;
    constexpr int NB = S::NB;
    constexpr int NQ = RB / 4;
    typedef typename vec_of<BV>::type bvec;

    __shared__ __align__(16) float lds[S::TOTAL];

    const int tid = threadIdx.x, lane = tid & 63;
    // uniform across the wave; saying so keeps the role branch and every
    // address derived from the wave index scalar
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int tiles = p.tiles_m * p.tiles_n;
    const int tile = blockIdx.x % tiles, split = blockIdx.x / tiles;
    const int tm = tile / p.tiles_n, tn = tile % p.tiles_n;
    const int64_t m = p.m, n = p.n, k = p.k;
    const int N = p.N, M = p.M, V = p.V;
    const int64_t q = n / V;
    const int64_t row0 = (int64_t)tm * S::ROWS, col0 = (int64_t)tn * S::COLS;

    // windows [gb, ge) of this workgroup, in stages of sw windows
    const int64_t G = k / M;
    const int64_t gps = (G + p.splits - 1) / p.splits;
    const int64_t gb = min64(G, (int64_t)split * gps), ge = min64(G, gb + gps);
    const int sw = p.sw;
    const int nst = (int)((ge - gb + sw - 1) / sw);
    // column blocks of the tile: [blk0, blk0 + qb) inside n
    const int64_t blk0 = col0 / V;
    const int qb = (int)(min64(q, (col0 + S::COLS - 1) / V + 1) - blk0);
    // compressed rows of stage s (0 past the last stage)
    auto stage_rows = [&](int s) { return (int)max64(0, min64(sw, ge - (gb + (int64_t)s * sw))) * N; };

    // Schedule (B_s: workgroup barrier; batch j: A_s and B_s of stage j and
    // X_s of stage j+1, in slot j % NB, X_s in slot (j+1) % (NB+1)):
    //   loaders:  X_s of stage 0 and batches 0 .. NB-2; then for each s: wait
    //             for batch s; B_s; batch s+NB-1
    //   compute:  for each s: B_s; read the offsets of stage s+1 and the
    //             operands of stage s; MFMAs of stage s
    // After B_s every compute wave is done with stage s-1, whose slot takes
    // batch s+NB-1.
    if (wave >= PS_NC) {
        // ---------------- loader waves ----------------
        // Loader l issues A row (pair) instructions l, l+NL, ..., Bc row
        // pieces l, l+NL, ... and offset-byte instructions l, l+NL, ...  The
        // lane part of each offset is fixed for the kernel; the row part is
        // one scalar per instruction, so an instruction costs a few scalar
        // operations.
        const int l = wave - PS_NC;
        constexpr int NA = S::IA / PS_NL, NBI = S::IB / PS_NL, NXI = (S::IX + PS_NL - 1) / PS_NL;
        const int nx = (S::IX - l + PS_NL - 1) / PS_NL;   // offset-byte instructions of this wave
        const int cnt = NA + NBI + nx;                     // DMA instructions of this wave per batch
        const int rows_valid = (int)min64(S::ROWS, m - row0);
        // rows past m fall outside the A resource and read zero.  Columns
        // past a partial last stage are read but never gathered.
        const __amdgpu_buffer_rsrc_t a_rsrc =
            make_rsrc(p.A + row0 * k, (uint32_t)((int64_t)rows_valid * k * 4));
        // lanes 0-31: the first row of a pair, lanes 32-63 the row H below
        const uint32_t a_lane = (uint32_t)(((lane >> 5) * S::H * k + 4 * (lane & 31)) * 4);
        // this loader's Bc piece is fixed (l % PB); columns past n get bit 31
        // (OOB), which stays past every buffer after a row offset is added
        const int64_t bcol = col0 + (S::PB > 1 ? l % S::PB : 0) * 256 + 4 * lane;
        const uint32_t b_lane = (uint32_t)(bcol * 4) | ((uint32_t)!(bcol < n) << 31);
        uint32_t x_lane[NXI];
#pragma unroll
        for (int ii = 0; ii < NXI; ++ii) {
            const int e = (l + PS_NL * ii) * 64 + lane;
            const int rho = e / S::QBMAX, lb = e % S::QBMAX;
            x_lane[ii] = rho < RB && lb < qb ? (uint32_t)((int64_t)rho * q + blk0 + lb) : OOB;
        }
        auto issue_x = [&](int s) {
            // offset bytes past the stage (or of a stage past the last) read zero
            const __amdgpu_buffer_rsrc_t x_rsrc =
                make_rsrc(p.idx + (gb + (int64_t)s * sw) * N * q, (uint32_t)((int64_t)stage_rows(s) * q));
            float *xb = lds + S::X_BASE + (s % (NB + 1)) * S::X_INTS;
#pragma unroll
            for (int ii = 0; ii < NXI; ++ii)
                if (ii < nx) lds_dma<1>(x_rsrc, xb + (l + PS_NL * ii) * 64, x_lane[ii]);
        };
        auto issue = [&](int s) {
            const int64_t g0 = gb + (int64_t)s * sw;
            const int rsn = stage_rows(s);
            const uint32_t a_col = (uint32_t)(g0 * M * 4);
            // rows of Bc past the stage fall outside this resource and read zero
            const __amdgpu_buffer_rsrc_t b_rsrc = make_rsrc(p.Bc + g0 * N * n, (uint32_t)((int64_t)rsn * n * 4));
            float *base = lds + (s % NB) * S::STAGE;
#pragma unroll
            for (int ii = 0; ii < NA; ++ii) {
                const int pr = l + PS_NL * ii;
                const int row = RT >= 2 ? 32 * (pr / 16) + pr % 16 : pr;   // first row of pair pr
                lds_dma<16>(a_rsrc, base + pr * S::AST, a_lane + (uint32_t)(row * k * 4) + a_col);
            }
            if (lane < S::LB) {
#pragma unroll
                for (int ii = 0; ii < NBI; ++ii) {
                    const int ib = l + PS_NL * ii;
                    const int rho = ib / S::PB, piece = ib % S::PB;
                    lds_dma<16>(b_rsrc, base + S::A_FLOATS + rho * S::BST + piece * 256,
                                b_lane + (uint32_t)(rho * n * 4));
                }
            }
            issue_x(s + 1);
        };
        issue_x(0);
        const int pre = nst < NB - 1 ? nst : NB - 1;
        for (int s = 0; s < pre; ++s) issue(s);
        for (int s = 0; s < nst; ++s) {
            // batch s has landed once at most the batches issued after it are
            // in flight: min(NB - 2, nst - 1 - s) of them
            const int after = nst - 1 - s < NB - 2 ? nst - 1 - s : NB - 2;
            vm_wait_le<0, (NB - 2) * S::CMAX>(after * cnt);
            ps_barrier();
            if (s + NB - 1 < nst) issue(s + NB - 1);
        }
        if (p.splits == 1) return;
        // split-k epilogue: every DMA has landed before LDS is reused
        __builtin_amdgcn_s_waitcnt(0);
        ps_barrier();
        ps_barrier();
    } else {
        // ---------------- compute waves ----------------
        const int r = lane & 15, kq = lane >> 4;
        const int c = wave;
        // local column block of each of this wave's column groups (a group
        // of CG columns lies inside one block: V is a multiple of CG)
        int lbk[CPW];
#pragma unroll
        for (int g = 0; g < CPW; ++g) lbk[g] = (int)((col0 + c * S::CW + g * S::CG) / V - blk0);
        // x / N for 0 <= x < 4096 as (x * invN) >> 20 (exact for N <= 256)
        const uint32_t invN = ((1u << 20) + N - 1) / N;
        auto read_x = [&](int s, int (&x)[NQ][CPW]) {
            const int *Xs = reinterpret_cast<const int *>(lds + S::X_BASE + (s % (NB + 1)) * S::X_INTS);
#pragma unroll
            for (int j = 0; j < NQ; ++j)
#pragma unroll
                for (int g = 0; g < CPW; ++g) x[j][g] = Xs[(4 * j + kq) * S::QBMAX + lbk[g]];
        };

        f32x4 acc[RT][CPW][BV];
#pragma unroll
        for (int t = 0; t < RT; ++t)
#pragma unroll
            for (int g = 0; g < CPW; ++g)
#pragma unroll
                for (int v = 0; v < BV; ++v) acc[t][g][v] = f32x4{0.f, 0.f, 0.f, 0.f};

        int xc[NQ][CPW];   // offsets of the current stage
        for (int s = 0; s < nst; ++s) {
            // this wave's reads of the previous stage are done before the barrier
            lds_drain();
            ps_barrier();
            if (s == 0) read_x(0, xc);
            // the next stage's offsets landed with this stage
            int xn[NQ][CPW];
            read_x(s + 1, xn);
            const float *As = lds + (s % NB) * S::STAGE + S::a_lane_base(r);
            const float *Bs = lds + (s % NB) * S::STAGE + S::A_FLOATS + c * S::CW + BV * r;
            const int rsn = stage_rows(s);
            // all of the stage's gathered A and Bc operands (rows past a
            // partial stage: zero in B_s, gather column 0), then its MFMAs
            float a[NQ][CPW][RT];
            bvec b[NQ][CPW];
#pragma unroll
            for (int j = 0; j < NQ; ++j) {
                const int ur = 4 * j + kq;
                const int wbase = (int)((ur * invN) >> 20) * M;
#pragma unroll
                for (int g = 0; g < CPW; ++g) {
                    const int ac = ur < rsn ? wbase + min(xc[j][g], M - 1) : 0;
                    b[j][g] = *reinterpret_cast<const bvec *>(Bs + ur * S::BST + g * S::CG);
#pragma unroll
                    for (int t = 0; t < RT; ++t) a[j][g][t] = As[S::a_row(t) + ac];
                }
            }
#pragma unroll
            for (int j = 0; j < NQ; ++j) {
                if (4 * j >= rsn) break;   // whole quads past a partial stage
#pragma unroll
                for (int g = 0; g < CPW; ++g)
#pragma unroll
                    for (int t = 0; t < RT; ++t)
#pragma unroll
                        for (int v = 0; v < BV; ++v)
                            acc[t][g][v] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                                a[j][g][t], lane_of<BV>(b[j][g], v), acc[t][g][v], 0, 0, 0);
            }
#pragma unroll
            for (int j = 0; j < NQ; ++j)
#pragma unroll
                for (int g = 0; g < CPW; ++g) xc[j][g] = xn[j][g];
        }

        // lane (r, kq) holds rows 16t + 4kq + e, columns c*CW + g*CG + BV*r + v
        if (p.splits == 1) {
#pragma unroll
            for (int g = 0; g < CPW; ++g) {
                const int64_t col = col0 + c * S::CW + g * S::CG + BV * r;
                if (col >= n) continue;
#pragma unroll
                for (int t = 0; t < RT; ++t)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int64_t row = row0 + 16 * t + 4 * kq + e;
                        if (row >= m) continue;
                        bvec v;
                        if constexpr (BV == 1) {
                            v = apply_epilogue(p.epi, acc[t][g][0][e], col);
                        } else {
#pragma unroll
                            for (int s = 0; s < BV; ++s) v[s] = apply_epilogue(p.epi, acc[t][g][s][e], col + s);
                        }
                        *reinterpret_cast<bvec *>(p.C + row * n + col) = v;
                    }
            }
            return;
        }
        // split-k: stage the tile in LDS once every wave is done with the ring
        lds_drain();
        ps_barrier();
#pragma unroll
        for (int g = 0; g < CPW; ++g)
#pragma unroll
            for (int t = 0; t < RT; ++t)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    bvec v;
                    if constexpr (BV == 1) {
                        v = acc[t][g][0][e];
                    } else {
#pragma unroll
                        for (int s = 0; s < BV; ++s) v[s] = acc[t][g][s][e];
                    }
                    *reinterpret_cast<bvec *>(lds + (16 * t + 4 * kq + e) * S::CST + c * S::CW + g * S::CG + BV * r) = v;
                }
        lds_drain();
        ps_barrier();
    }
    // split-k with a workspace: the staged tile goes to this workgroup's
    // slice; a second kernel adds the slices into C
    if (p.ws) {
        auto part = [&](int e) { return lds[(e / S::COLS) * S::CST + e % S::COLS]; };
        splitk_store<S::ROWS, S::COLS, PS_NT>(part, p.ws, tile, split, p.splits);
        return;
    }
    // split-k: every thread adds consecutive outputs of the staged tile
    // (coalesced atomics)
    for (int e = tid; e < S::ROWS * S::COLS; e += PS_NT) {
        const int rr = e / S::COLS, cc = e % S::COLS;
        const int64_t row = row0 + rr, col = col0 + cc;
        if (row < m && col < n) unsafeAtomicAdd(p.C + row * n + col, lds[rr * S::CST + cc]);
    }
}

template <int RT, int BV, int CPW, int RB>
hipError_t launch(const StreamArgs &a, hipStream_t stream)
{
    const unsigned grid = (unsigned)a.tiles_m * (unsigned)a.tiles_n * (unsigned)a.splits;
    hipLaunchKernelGGL((nm_stream_kernel<RT, BV, CPW, RB>), dim3(grid), dim3(PS_NT), 0, stream, a);
    return hipGetLastError();
}

}  // namespace

int stream_rows(int RT) { return 16 * RT; }
int stream_cols(int BV, int CPW) { return PS_NC * 16 * BV * CPW; }
int stream_stage_cols() { return PS_KS; }

// Instantiated (RT, BV, CPW, RB).
#define NMSPMM_STREAM_VARIANTS(X)                                                              \
    X(1, 1, 1, 16) X(1, 2, 1, 16) X(1, 4, 1, 16) X(1, 2, 1, 32) X(1, 4, 1, 32) X(1, 1, 1, 64) \
    X(2, 1, 1, 16) X(2, 2, 1, 16) X(2, 4, 1, 16) X(2, 2, 1, 32) X(2, 1, 1, 32)                \
    X(4, 1, 1, 16) X(4, 2, 1, 16) X(2, 2, 2, 16) X(1, 2, 2, 16)

bool stream_has(int RT, int BV, int CPW, int RB)
{
#define NM_PS_HAS(rt, bv, cpw, rb) \
    if (RT == rt && BV == bv && CPW == cpw && RB == rb) return true;
    NMSPMM_STREAM_VARIANTS(NM_PS_HAS)
#undef NM_PS_HAS
    return false;
}

hipError_t launch_stream(int RT, int BV, int CPW, int RB, const StreamArgs &a, hipStream_t stream)
{
#define NM_PS_LAUNCH(rt, bv, cpw, rb) \
    if (RT == rt && BV == bv && CPW == cpw && RB == rb) return launch<rt, bv, cpw, rb>(a, stream);
    NMSPMM_STREAM_VARIANTS(NM_PS_LAUNCH)
#undef NM_PS_LAUNCH
    return hipErrorInvalidValue;
}

}  // namespace nmspmm

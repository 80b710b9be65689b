// Direct-gather kernel for short products (m <= 128 rows), run through a
// caller-owned workspace.
//
// Eq. 1 gathers, for compressed row u and column block b, the column
// (u/N)*M + D[u][b] of A.  In row-major A the m values of one column lie k
// floats apart, so a gather touches m cache lines for m useful floats, and
// the streaming kernels instead stage whole slabs of A in LDS (the
// non-packing load of Sec. III-C.1).  Here a first pass writes A transposed
// into the workspace (At: one row of 16*RT floats per column of A, rows past
// m zero), so that the values one compressed row needs are contiguous, and
// precomputes for every (b, u) the byte offset of that At row (the
// per-block column indices of Sec. III-C.1, laid out u-contiguous per
// block).  The second pass then gathers At rows straight into registers.
//
// Strip kernel: a workgroup owns all rows (16*RT) x 16*CT columns of C (one
// strip inside one column block, V a multiple of 16*CT) and, with split-k, a
// range of quads (4 consecutive compressed rows, the K of
// v_mfma_f32_16x16x4_f32).  Its NW waves take that range's trips of D quads
// in turn and each streams its quads through a ring of D quads in flight in
// registers: per quad a
// lane loads one offset, RT At floats (one per row tile t, see c_row) and CT
// consecutive Bc floats (columns CT*(l%16)+s, one per column tile s), and
// issues RT*CT MFMAs.  No LDS and no barrier in the
// loop; the waves' partial strips are summed through LDS at the end, in a
// fixed order.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "nmspmm_gather.h"

namespace nmspmm {

namespace {

constexpr int TK = 32;  // columns of A per transposition block
constexpr int OU = 16;  // compressed rows per offset block (x 64 column blocks)

// First pass.  Blocks [0, tblocks) transpose TK columns of A each through
// LDS, in 16-byte pieces both ways when k is a multiple of 4 and A 16-byte
// aligned (VEC; measured on MI355X at 128 x 8192 x 8192: 6.07 -> 5.65 us per
// pass), else float by float; the others turn OU compressed rows x 64 column
// blocks of D into At byte offsets (offsets >= M, outside the contract, are
// clamped to M-1 so that every gather stays inside At).  Every thread issues
// all its loads before its first LDS store.
template <int ROWS, bool VEC>
__global__ __launch_bounds__(256) void nm_gather_prep_kernel(const float *__restrict__ A,
                                                             const uint8_t *__restrict__ idx,
                                                             float *__restrict__ At,
                                                             int32_t *__restrict__ off, int m, int k,
                                                             int w, int q, int N, int M, int tblocks,
                                                             int ublocks)
{
    __shared__ float t[ROWS * (TK + 1)];
    __shared__ int32_t o[64 * (OU + 1)];
    // row half blockIdx.y (its own At of ROWS-float rows; the offset blocks
    // run once, in half 0)
    const int h = (int)blockIdx.y;
    if (h > 0 && (int)blockIdx.x >= tblocks) return;
    A += (int64_t)h * ROWS * k;
    At += (int64_t)h * k * ROWS;
    m = max(0, min(ROWS, m - h * ROWS));
    if (VEC && (int)blockIdx.x < tblocks) {
        // ROWS x TK/4 pieces of 4 columns in, TK x ROWS/4 pieces of 4 rows out
        constexpr int PIECES = ROWS * TK / 4, PER = (PIECES + 255) / 256;
        const int c0 = (int)blockIdx.x * TK;
        f32x4 v[PER];
#pragma unroll
        for (int x = 0; x < PER; ++x) {
            const int e = threadIdx.x + 256 * x, i = e / (TK / 4), c = 4 * (e % (TK / 4));
            v[x] = (e < PIECES && i < m && c0 + c < k)
                       ? *reinterpret_cast<const f32x4 *>(A + (int64_t)i * k + c0 + c)
                       : f32x4{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int x = 0; x < PER; ++x) {
            const int e = threadIdx.x + 256 * x, i = e / (TK / 4), c = 4 * (e % (TK / 4));
            if (e < PIECES)
#pragma unroll
                for (int j = 0; j < 4; ++j) t[i * (TK + 1) + c + j] = v[x][j];
        }
        __syncthreads();
#pragma unroll
        for (int x = 0; x < PER; ++x) {
            const int e = threadIdx.x + 256 * x, c = e / (ROWS / 4), i = 4 * (e % (ROWS / 4));
            if (e < PIECES && c0 + c < k)
                *reinterpret_cast<f32x4 *>(At + (int64_t)(c0 + c) * ROWS + i) =
                    f32x4{t[i * (TK + 1) + c], t[(i + 1) * (TK + 1) + c], t[(i + 2) * (TK + 1) + c],
                          t[(i + 3) * (TK + 1) + c]};
        }
        return;
    }
    if ((int)blockIdx.x < tblocks) {
        constexpr int PER = ROWS * TK / 256;
        const int c0 = (int)blockIdx.x * TK;
        float v[PER];
#pragma unroll
        for (int x = 0; x < PER; ++x) {
            const int e = threadIdx.x + 256 * x, i = e / TK, c = e % TK;
            v[x] = (i < m && c0 + c < k) ? A[(int64_t)i * k + c0 + c] : 0.f;
        }
#pragma unroll
        for (int x = 0; x < PER; ++x) {
            const int e = threadIdx.x + 256 * x;
            t[(e / TK) * (TK + 1) + e % TK] = v[x];
        }
        __syncthreads();
#pragma unroll
        for (int x = 0; x < PER; ++x) {
            const int e = threadIdx.x + 256 * x, c = e / ROWS, i = e % ROWS;
            if (c0 + c < k) At[(int64_t)(c0 + c) * ROWS + i] = t[i * (TK + 1) + c];
        }
        return;
    }
    constexpr int PER = OU * 64 / 256;
    const int ob = (int)blockIdx.x - tblocks;
    const int u0 = (ob % ublocks) * OU, b0 = (ob / ublocks) * 64;
    int d[PER];
#pragma unroll
    for (int x = 0; x < PER; ++x) {
        const int e = threadIdx.x + 256 * x, u = u0 + e / 64, b = b0 + e % 64;
        d[x] = (u < w && b < q) ? (int)idx[(int64_t)u * q + b] : 0;
    }
#pragma unroll
    for (int x = 0; x < PER; ++x) {
        const int e = threadIdx.x + 256 * x, du = e / 64, u = u0 + du;
        o[(e % 64) * (OU + 1) + du] = ((u / N) * M + min(d[x], M - 1)) * (ROWS * 4);
    }
    __syncthreads();
#pragma unroll
    for (int x = 0; x < PER; ++x) {
        const int e = threadIdx.x + 256 * x, db = e / OU, du = e % OU;
        const int u = u0 + du, b = b0 + db;
        if (u < w && b < q) off[(int64_t)b * w + u] = o[db * (OU + 1) + du];
    }
}

// A lane's At floats: RH = min(RT, 4) consecutive rows per 16-byte load, and
// RT/RH such loads, half h covering rows [16*RH*h, 16*RH*(h+1)) of the At row
// (so that each load reads one contiguous piece of the row).  MFMA row tile t,
// MFMA row i then holds row  (t/RH)*16*RH + RH*i + t%RH  of C.
template <int RT> constexpr int rows_per_load() { return RT < 4 ? RT : 4; }
template <int RT>
__device__ __forceinline__ int c_row(int t, int i)
{
    constexpr int RH = rows_per_load<RT>();
    return (t / RH) * 16 * RH + RH * i + t % RH;
}

template <int RT> struct AOp;
template <> struct AOp<1> { float v[1]; };
template <> struct AOp<2> { float v[2]; };
template <> struct AOp<4> { float v[4]; };
template <> struct AOp<8> { float v[8]; };

template <int RT>
__device__ __forceinline__ void load_a(AOp<RT> &a, __amdgpu_buffer_rsrc_t rs, uint32_t voff)
{
    if constexpr (RT == 1) {
        a.v[0] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, (int)voff, 0, 0));
    } else if constexpr (RT == 2) {
        const f32x2 x = __builtin_bit_cast(f32x2, __builtin_amdgcn_raw_buffer_load_b64(rs, (int)voff, 0, 0));
        a.v[0] = x[0];
        a.v[1] = x[1];
    } else {
#pragma unroll
        for (int h = 0; h < RT / 4; ++h) {
            const f32x4 x =
                __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, (int)(voff + 256 * h), 0, 0));
#pragma unroll
            for (int i = 0; i < 4; ++i) a.v[4 * h + i] = x[i];
        }
    }
}

template <int CT> struct BOp;
template <> struct BOp<2> { float v[2]; };
template <> struct BOp<4> { float v[4]; };

// Bc is read once: up to 64 rows its loads carry the non-temporal hint (cache
// policy bit 1), so that the streamed lines leave L2 to the At rows, which fit
// in one XCD's 4 MB L2 up to there (2 MB at 64 rows x k = 8192).  Measured on
// MI355X at k = n = 8192, 4:32: 64 rows 22.1 -> 21.7 us; at 128 rows (4 MB of
// At) it measured 0.5 us slower, and those loads keep the default policy.
template <int CT, int AUX>
__device__ __forceinline__ void load_b(BOp<CT> &b, __amdgpu_buffer_rsrc_t rs, uint32_t voff, uint32_t soff)
{
    if constexpr (CT == 2) {
        const f32x2 x =
            __builtin_bit_cast(f32x2, __builtin_amdgcn_raw_buffer_load_b64(rs, (int)voff, (int)soff, AUX));
        b.v[0] = x[0];
        b.v[1] = x[1];
    } else {
        const f32x4 x =
            __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, (int)voff, (int)soff, AUX));
#pragma unroll
        for (int i = 0; i < 4; ++i) b.v[i] = x[i];
    }
}

template <int RT, int CT>
__device__ __forceinline__ void mma_quad(f32x4 (&acc)[RT][CT], const AOp<RT> &a, const BOp<CT> &b)
{
#pragma unroll
    for (int t = 0; t < RT; ++t)
#pragma unroll
        for (int s = 0; s < CT; ++s)
            acc[t][s] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v[t], b.v[s], acc[t][s], 0, 0, 0);
}

template <int RT, int CT, int NW>
struct GShape {
    static constexpr int ROWS = 16 * RT, COLS = 16 * CT;
    static constexpr int RST = COLS + 1;                 // LDS row stride of a partial strip
    static constexpr int TILE = ROWS * RST;
    // partial strips held in LDS at once (a power of two dividing NW); the
    // waves beyond them add into the held ones, in wave order
    static constexpr int FIT = (120 * 1024 / 4) / TILE;
    static constexpr int G = FIT >= NW ? NW : FIT >= 4 ? 4 : FIT >= 2 ? 2 : 1;
};

template <int RT, int CT, int NW, int D>
__global__ __launch_bounds__(NW * 64) void nm_gather_kernel(
    const float *__restrict__ At, const int32_t *__restrict__ off, const float *__restrict__ Bc,
    float *__restrict__ C, float *__restrict__ part, int m, int64_t n, int k, int w, int V, int strips,
    int splits, int halves, Epilogue epi)
{
    using S = GShape<RT, CT, NW>;
    constexpr int ROWS = S::ROWS, COLS = S::COLS, RST = S::RST;
    constexpr int BC_AUX = RT <= 4 ? 2 : 0;
    __shared__ float red[S::G * S::TILE];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    // Workgroups are dispatched round-robin over the 8 XCDs: renumber them so
    // that consecutive strips, which gather the same At rows when they share a
    // column block, run on one XCD and share its L2.
    const int nwg = gridDim.x, pid = blockIdx.x;
    const int xcd = pid % 8, local = pid / 8, full = nwg / 8, rem = nwg % 8;
    const int logical = xcd < rem ? xcd * (full + 1) + local : rem * (full + 1) + (xcd - rem) * full + local;
    // the row halves of one strip are consecutive (one XCD: they share its
    // Bc lines in L2); each has its own At of ROWS-float rows
    const int h = logical % halves, rest = logical / halves;
    const int split = rest / strips, strip = rest - split * strips;
    At += (int64_t)h * k * ROWS;
    C += (int64_t)h * ROWS * n;
    m = max(0, min(ROWS, m - h * ROWS));
    const int64_t j0 = (int64_t)strip * COLS;
    const int b = (int)(j0 / V);
    const int nquads = (w + 3) / 4;
    const int qs = (int)((int64_t)split * nquads / splits);
    const int qe = (int)((int64_t)(split + 1) * nquads / splits);
    const int nq = qe - qs;
    // trips of D quads are dealt to the waves in turn (wave v takes trips v,
    // v + NW, ...), so that at any time the waves stream one band of Bc
    const int ntrips = (nq + D - 1) / D;

    const int r = lane & 15, kq = lane >> 4;
    // The split's Bc rows only: quads past its range (the ring loads one trip
    // ahead) and rows past w read zero and add nothing.  Offsets past w read
    // zero too, which gathers At row 0, in bounds.
    const int64_t u_lo = min64(4 * (int64_t)qs, w), u_hi = min64(4 * (int64_t)qe, w);
    const auto rs_at = make_rsrc(At, (uint32_t)k * ROWS * 4);
    const auto rs_off = make_rsrc(off + (int64_t)b * w + u_lo, (uint32_t)(w - u_lo) * 4);
    const auto rs_bc = make_rsrc(Bc + u_lo * n + j0, (uint32_t)(max64(u_hi - u_lo, 0) * n * 4));
    const uint32_t lane_off = kq * 4;
    const uint32_t lane_bc = (uint32_t)((kq * n + CT * r) * 4);
    const uint32_t lane_at = r * rows_per_load<RT>() * 4;
    const uint32_t quad_bc = (uint32_t)(16 * n);   // bytes of 4 Bc rows

    f32x4 acc[RT][CT];
#pragma unroll
    for (int t = 0; t < RT; ++t)
#pragma unroll
        for (int s = 0; s < CT; ++s) acc[t][s] = f32x4{0.f, 0.f, 0.f, 0.f};

    // Ring of D slots: after trip t, slot j holds the operands of quad
    // t*D + j and the offset of quad (t+1)*D + j.  Trip 0 only loads; every
    // later trip multiplies the previous trip's quads and loads its own.
    AOp<RT> av[D];
    BOp<CT> bv[D];
    uint32_t ov[D];
    // The first trip's offsets, each slot issued as the loop issues it (A, Bc,
    // offset; the A and Bc loads out of range, reading zero), so that the
    // pending loads on entry line up with those of a trip and the wait counts
    // at the loop head stay exact.
#pragma unroll
    for (int j = 0; j < D; ++j) {
        load_a<RT>(av[j], rs_at, OOB + 1024 * j);   // distinct offsets: no two loads merged
        load_b<CT, BC_AUX>(bv[j], rs_bc, OOB + 64 * j, 0);
        ov[j] = __builtin_amdgcn_raw_buffer_load_b32(rs_off, (int)lane_off, (wave * D + j) * 16, 0);
        __builtin_amdgcn_sched_barrier(0);
    }
    const int trips = ntrips > wave ? (ntrips - wave + NW - 1) / NW : 0;
    // one loop, not peeled: a peeled first trip behind its own branch lets
    // the compiler sink its loads, and the wait counts at the loop head
    // become conservative
#pragma clang loop unroll(disable)
    for (int t = 0; t <= trips; ++t) {
#pragma unroll
        for (int j = 0; j < D; ++j) {
            // quads past the wave's range read zero: skip their MFMAs
            if (t > 0 && ((t - 1) * NW + wave) * D + j < nq) mma_quad<RT, CT>(acc, av[j], bv[j]);
            const int qn = (t * NW + wave) * D + j;
            load_a<RT>(av[j], rs_at, ov[j] + lane_at);
            load_b<CT, BC_AUX>(bv[j], rs_bc, lane_bc, qn * quad_bc);
            ov[j] = __builtin_amdgcn_raw_buffer_load_b32(rs_off, (int)lane_off, (qn + NW * D) * 16, 0);
            // keep each slot's loads right after its MFMAs: gathered to the
            // end of the unrolled body, they would be waited for at once
            __builtin_amdgcn_sched_barrier(0);
        }
    }

    // partial strips of the waves, summed in a fixed order: G held in LDS,
    // the waves beyond them adding into the held ones round by round
    float *mine = red + (wave % S::G) * S::TILE;
#pragma unroll 1
    for (int round = 0; round < NW / S::G; ++round) {
        if (wave / S::G == round) {
#pragma unroll
            for (int t = 0; t < RT; ++t)
#pragma unroll
                for (int s = 0; s < CT; ++s)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        float &x = mine[c_row<RT>(t, 4 * kq + i) * RST + CT * r + s];
                        x = round == 0 ? acc[t][s][i] : x + acc[t][s][i];
                    }
        }
        __syncthreads();
    }
    for (int e = threadIdx.x; e < ROWS * COLS; e += NW * 64) {
        const int row = e / COLS, col = e % COLS;
        float sum = red[row * RST + col];
#pragma unroll
        for (int x = 1; x < S::G; ++x) sum += red[x * S::TILE + row * RST + col];
        if (splits == 1) {
            if (row < m) C[(int64_t)row * n + j0 + col] = apply_epilogue(epi, sum, j0 + col);
        } else {
            part[((int64_t)strip * splits + split) * (ROWS * COLS) + e] = sum;
        }
    }
}

template <int RT, int CT, int NW, int D>
hipError_t launch_cfg(const GatherArgs &a, hipStream_t stream)
{
    constexpr int ROWS = 16 * RT, COLS = 16 * CT;
    GatherCfg cfg{RT, CT, NW, D};
    cfg.H = a.halves;
    const int w = (int)(a.k / a.M * a.N), q = (int)(a.n / a.V), strips = (int)(a.n / COLS);
    const GatherLayout L = gather_layout(cfg, a.n, a.k, a.N, a.M, a.V, a.splits);
    char *base = static_cast<char *>(a.ws);
    float *At = reinterpret_cast<float *>(base + L.at);
    int32_t *off = reinterpret_cast<int32_t *>(base + L.off);
    float *part = a.splits > 1 ? reinterpret_cast<float *>(base + L.part) : nullptr;
    const int tblocks = (int)((a.k + TK - 1) / TK), ublocks = (w + OU - 1) / OU, bblocks = (q + 63) / 64;
    const int H = a.splits == 1 ? max(1, a.halves) : 1;
    if (a.k % 4 == 0 && reinterpret_cast<uintptr_t>(a.A) % 16 == 0)
        hipLaunchKernelGGL((nm_gather_prep_kernel<ROWS, true>), dim3((unsigned)(tblocks + ublocks * bblocks), H),
                           dim3(256), 0, stream, a.A, a.idx, At, off, (int)a.m, (int)a.k, w, q, a.N, a.M, tblocks,
                           ublocks);
    else
        hipLaunchKernelGGL((nm_gather_prep_kernel<ROWS, false>), dim3((unsigned)(tblocks + ublocks * bblocks), H),
                           dim3(256), 0, stream, a.A, a.idx, At, off, (int)a.m, (int)a.k, w, q, a.N, a.M, tblocks,
                           ublocks);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((nm_gather_kernel<RT, CT, NW, D>), dim3((unsigned)(strips * a.splits * H)), dim3(NW * 64),
                       0, stream, At, off, a.Bc, a.C, part, (int)a.m, a.n, (int)a.k, w, a.V, strips, a.splits, H,
                       a.epi);
    return hipGetLastError();
}

// Instantiated configurations: {RT, CT, NW, D}.
#define NM_GATHER_CONFIGS(X)                                                                            \
    X(1, 2, 8, 4) X(1, 2, 8, 8) X(1, 4, 8, 4) X(1, 4, 4, 8)                                             \
    X(2, 2, 8, 4) X(2, 2, 8, 8) X(2, 4, 8, 4)                                                           \
    X(4, 2, 8, 4) X(4, 2, 8, 3) X(4, 2, 8, 8) X(4, 4, 8, 4) X(4, 4, 4, 8)                               \
    X(8, 2, 4, 4) X(8, 2, 4, 8) X(8, 2, 8, 4) X(8, 4, 4, 4) X(8, 4, 4, 6)

}  // namespace

int gather_rows(int RT) { return 16 * RT; }

bool gather_has(const GatherCfg &c)
{
#define NM_GATHER_HAS(RT_, CT_, NW_, D_) \
    if (c.RT == RT_ && c.CT == CT_ && c.NW == NW_ && c.D == D_) return true;
    NM_GATHER_CONFIGS(NM_GATHER_HAS)
#undef NM_GATHER_HAS
    return false;
}

GatherLayout gather_layout(const GatherCfg &c, int64_t n, int64_t k, int N, int M, int V, int splits)
{
    const int64_t halves = splits == 1 ? std::max(1, c.H) : 1;
    auto up = [](int64_t x) { return (x + 255) / 256 * 256; };
    const int64_t w = k / M * N, q = n / V, strips = n / (16 * c.CT);
    GatherLayout L;
    L.at = 0;
    L.off = up(halves * k * 16 * c.RT * 4);
    L.part = L.off + up(q * w * 4);
    L.total = L.part + (splits > 1 ? up(strips * splits * 16 * c.RT * 16 * c.CT * 4) : 0);
    return L;
}

hipError_t launch_gather(const GatherCfg &c, const GatherArgs &a, hipStream_t stream)
{
#define NM_GATHER_LAUNCH(RT_, CT_, NW_, D_) \
    if (c.RT == RT_ && c.CT == CT_ && c.NW == NW_ && c.D == D_) return launch_cfg<RT_, CT_, NW_, D_>(a, stream);
    NM_GATHER_CONFIGS(NM_GATHER_LAUNCH)
#undef NM_GATHER_LAUNCH
    return hipErrorInvalidValue;
}

}  // namespace nmspmm

// Tiled fp32-MFMA kernel for vector-wise N:M SpMM on gfx950 (device code,
// included by the per-shape instantiation units).
//
// One workgroup owns a BM x BN tile of C (and, with split-k, one slice of the
// k range).  It walks k in stages of KA = 32 columns of A: 32/M windows and
// RS = (32/M)*N compressed rows, padded to RST = 4*NQ rows (MFMA K = 4).
// Each stage is brought into a ring of P LDS slots (Sec. III-B.1's blocking;
// Sec. III-C.2's pipeline, deepened from two buffers to P so that several
// stages of HBM latency are in flight):
//   A_s : the BM x KA slab of A, row-major, 128 bytes per row.  The whole
//         slab is staged (the non-packing load of Sec. III-C.1): with random
//         per-block patterns nearly every column is needed by some block of
//         the tile.  16-byte chunk j of row i sits at chunk position
//         j ^ ((i >> 1) & 7), so that sixteen consecutive rows of one column
//         fall in distinct LDS banks when the gather reads them.
//   B_s : the RST x BN slab of Bc, row-major (padding rows are zero).
//   X_s : the RST x (BN/V) offset bytes of D, one zero-extended dword each.
// All three are filled by buffer->LDS DMA (no register staging); a lane picks
// the global address whose data must land at its fixed LDS position, which
// is how the swizzle is applied.  Out-of-range lanes (ragged m, n, k tails,
// padding rows) read zero.  Every wave issues the same number of DMA
// instructions per stage, so "stage s has landed" is a counted vmcnt wait
// followed by one barrier; the same barrier frees the slot of stage s-1 for
// the DMA of stage s+P-1.
//
// Contraction: v_mfma_f32_16x16x4_f32 (fp32 in, fp32 accumulate).  Lane l
// supplies A[l%16][l/16] and B[l/16][l%16] and receives D[4*(l/16)+v][l%16]
// in element v.  The K index l/16 selects one of four consecutive compressed
// rows, each with its own gather offset (the index prefetch of Sec. III-C.2
// turns it into an LDS address once per stage); the 16 columns of one MFMA
// lie in a column group of CG = 16*BV columns inside a single column block,
// so they share one gather.  A lanes read output row l%16 of a 16-row chunk,
// B lanes read columns BV*(l%16)+s, s < BV (BV MFMAs per A read).  The
// LDS->register fetch of quad q+1 is issued before the MFMAs of quad q (the
// register double buffer of Sec. III-C.2).
#ifndef NMSPMM_TILED_H
#define NMSPMM_TILED_H

#include <hip/hip_runtime.h>

#include <cstdint>

namespace nmspmm {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;

template <int W> struct vec_of;
template <> struct vec_of<1> { typedef float type; };
template <> struct vec_of<2> { typedef f32x2 type; };
template <> struct vec_of<4> { typedef f32x4 type; };

template <int W>
__device__ __forceinline__ float lane_of(const typename vec_of<W>::type &v, int i)
{
    if constexpr (W == 1) return v; else return v[i];
}

constexpr int LDS_CAPACITY = 160 * 1024;
constexpr int KA = 32;            // A columns per stage
constexpr int A_ROW_BYTES = KA * 4;

template <int BM_, int BN_, int WM_, int WN_>
struct TileCfg {
    static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_;
    static constexpr int NW = (BM / WM) * (BN / WN);
    static constexpr int NT = NW * 64;
    static constexpr int NRC = WM / 16;         // 16-row MFMA chunks per wave
    static_assert(WM % 16 == 0 && BM % WM == 0 && BN % WN == 0, "tile shape");
};

// Per-instantiation constants (tile shape x column-group width x quads per stage).
template <class T, int BV, int NQ>
struct Shape {
    static constexpr int CG = 16 * BV;
    static constexpr int NCG = T::WN / CG;
    static constexpr int RST = 4 * NQ;                 // padded rows per stage
    static constexpr int QBMAX = T::BN / CG;           // column blocks per tile, at most
    static constexpr int A_BYTES = T::BM * A_ROW_BYTES;
    static constexpr int B_BYTES = RST * T::BN * 4;
    static constexpr int X_BYTES = T::NT * 4;
    static constexpr int STAGE_BYTES = A_BYTES + B_BYTES + X_BYTES;
    // DMA instruction width (bytes per lane) and count per wave per stage
    static constexpr int A_LANE = A_BYTES / T::NT;
    static constexpr int A_W = A_LANE % 16 == 0 ? 16 : 4;
    static constexpr int A_CNT = A_LANE / A_W;
    static constexpr int B_LANE = B_BYTES / T::NT;
    static constexpr int B_W = B_LANE % 16 == 0 ? 16 : 4;
    static constexpr int B_CNT = B_LANE / B_W;
    static constexpr int LOADS = A_CNT + B_CNT + 1;    // DMA instructions per wave per stage
    static constexpr int P_RAW = LDS_CAPACITY / STAGE_BYTES;
    static constexpr int P = P_RAW > 6 ? 6 : P_RAW;    // ring depth
    static constexpr bool FITS = P >= 2 && T::WN % CG == 0 && RST * QBMAX <= T::NT &&
                                 A_BYTES % T::NT == 0 && B_BYTES % T::NT == 0 &&
                                 A_LANE % 4 == 0 && B_LANE % 4 == 0 && A_CNT >= 1 &&
                                 B_CNT >= 1 && (P - 1) * LOADS < 64;
};

struct TiledArgs {
    const float *A;
    const float *Bc;
    const uint8_t *idx;
    float *C;
    int64_t m, n, k;
    int N, M, V;
    int RS;          // real compressed rows per stage, (32/M)*N
    int stages;      // ceil((k/M) / (32/M))
    int splits;      // split-k factor (>1: atomic accumulation into a zeroed C)
    int tiles_m, tiles_n;
};

// Workgroups are dispatched round-robin over the 8 XCDs.  Renumber them so
// that consecutive logical ids run on one XCD (and share its L2), then walk
// the tiles of one k-split in groups of GROUP_M tile rows, column-major inside
// a group, so that the workgroups of one XCD share A rows and Bc columns.
__device__ __forceinline__ void map_tile(int pid, int nwg, int tiles_m, int tiles_n, int &tm,
                                         int &tn, int &split)
{
    constexpr int NXCD = 8, GROUP_M = 4;
    const int xcd = pid % NXCD, local = pid / NXCD;
    const int full = nwg / NXCD, rem = nwg % NXCD;
    const int logical = xcd < rem ? xcd * (full + 1) + local
                                  : rem * (full + 1) + (xcd - rem) * full + local;
    const int ntiles = tiles_m * tiles_n;
    split = logical / ntiles;
    const int t = logical - split * ntiles;
    const int per_group = GROUP_M * tiles_n;
    const int group = t / per_group;
    const int first_m = group * GROUP_M;
    const int gm = min(tiles_m - first_m, GROUP_M);
    const int in_group = t - group * per_group;
    tm = first_m + in_group % gm;
    tn = in_group / gm;
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base, uint32_t bytes)
{
    // raw buffer, 32-bit dwords; accesses at offsets >= bytes read zero
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes,
                                             0x00020000);
}

constexpr uint32_t OOB = 0x80000000u;  // an offset past every buffer used here

// One buffer->LDS DMA instruction: lane l's W bytes from byte offset `off`
// of the buffer land at dst + l*W.
// (The width is spelled as a literal in each branch: the builtin needs an
// integer constant that is not template-dependent.)
template <int W>
__device__ __forceinline__ void lds_dma(__amdgpu_buffer_rsrc_t rsrc, void *dst, uint32_t off)
{
    static_assert(W == 1 || W == 4 || W == 16, "DMA width");
    if constexpr (W == 16)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void *)dst, 16, (int)off, 0, 0, 0);
    else if constexpr (W == 4)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void *)dst, 4, (int)off, 0, 0, 0);
    else
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void *)dst, 1, (int)off, 0, 0, 0);
}

// Wait until at most `later` DMA instructions of this wave are outstanding.
template <int LOADS, int PM2>
__device__ __forceinline__ void wait_vm(int later_stages)
{
    // s_waitcnt simm16 on gfx9: vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt[5:4]<<14;
    // expcnt and lgkmcnt are left at their maxima (no wait).
#define NMSPMM_VM(c) __builtin_amdgcn_s_waitcnt(((c) & 15) | (7 << 4) | (15 << 8) | (((c) >> 4) << 14))
    static_assert(PM2 <= 4, "ring depth");
    switch (later_stages) {
    case 0: NMSPMM_VM(0); break;
    case 1: NMSPMM_VM(1 * LOADS); break;
    case 2: if constexpr (PM2 >= 2) NMSPMM_VM(2 * LOADS); break;
    case 3: if constexpr (PM2 >= 3) NMSPMM_VM(3 * LOADS); break;
    default: if constexpr (PM2 >= 4) NMSPMM_VM(4 * LOADS); break;
    }
#undef NMSPMM_VM
}

// Workgroup barrier without a memory fence: LDS visibility is established by
// the explicit vmcnt / lgkmcnt waits; the empty asm keeps the compiler from
// moving memory accesses across it.
__device__ __forceinline__ void block_sync()
{
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt((15) | (7 << 4) | (0 << 8) | (3 << 14));  // lgkmcnt(0)
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

template <class T, int BV, int NQ>
__global__ __launch_bounds__(T::NT) void nm_tiled_kernel(TiledArgs p)
{
    using S = Shape<T, BV, NQ>;
    constexpr int BM = T::BM, BN = T::BN, WM = T::WM, WN = T::WN, NW = T::NW, NRC = T::NRC;
    constexpr int CG = S::CG, NCG = S::NCG, RST = S::RST, P = S::P, LOADS = S::LOADS;
    typedef typename vec_of<BV>::type bvec;

    __shared__ __align__(16) unsigned char lds[P * S::STAGE_BYTES];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    int tm, tn, split;
    map_tile(blockIdx.x, gridDim.x, p.tiles_m, p.tiles_n, tm, tn, split);
    const int64_t row0 = (int64_t)tm * BM, col0 = (int64_t)tn * BN;
    const int64_t m = p.m, n = p.n, k = p.k;
    const int N = p.N, M = p.M, V = p.V, RS = p.RS;
    const int64_t w = (k / M) * N, q = n / V;
    const int64_t b_first = col0 / V;
    const int QB = BN >= V ? BN / V : 1;

    const int sps = (p.stages + p.splits - 1) / p.splits;
    const int s_begin = split * sps;
    const int s_end = min(p.stages, s_begin + sps);
    if (p.splits > 1 && s_begin >= s_end) return;  // uniform over the workgroup
    const int nst = max(s_end - s_begin, 0);

    const int wm = wave / (BN / WN), wn = wave % (BN / WN);
    int blk[NCG];
#pragma unroll
    for (int cg = 0; cg < NCG; ++cg) blk[cg] = (int)((col0 + wn * WN + cg * CG) / V - b_first);

    // ---- per-lane DMA source offsets that do not change between stages ----
    const int rows_valid = (int)min<int64_t>(BM, m - row0);
    const __amdgpu_buffer_rsrc_t a_rsrc =
        make_rsrc(p.A + row0 * k, (uint32_t)((int64_t)rows_valid * k * 4));
    uint32_t a_off[S::A_CNT];      // byte offset of this lane's A piece, relative to column kc0
    int a_col[S::A_CNT];           // its first column inside the stage (for the k tail)
#pragma unroll
    for (int i = 0; i < S::A_CNT; ++i) {
        const int pos = ((i * NW + wave) * 64 + lane) * S::A_W;   // byte position in A_s
        const int row = pos / A_ROW_BYTES, inrow = pos % A_ROW_BYTES;
        const int chunk = (inrow >> 4) ^ ((row >> 1) & 7);
        const int colb = chunk * 16 + (inrow & 15);
        a_col[i] = colb / 4;
        a_off[i] = (uint32_t)((int64_t)row * k * 4 + colb);
    }
    uint32_t b_off[S::B_CNT];
    bool b_ok[S::B_CNT];
#pragma unroll
    for (int i = 0; i < S::B_CNT; ++i) {
        const int pos = ((i * NW + wave) * 64 + lane) * S::B_W;   // byte position in B_s
        const int ul = pos / (BN * 4), col = (pos % (BN * 4)) / 4;
        b_ok[i] = col0 + col < n;
        b_off[i] = (uint32_t)(((int64_t)ul * n + col0 + col) * 4);
    }
    const int x_ul = tid / QB, x_bl = tid % QB;
    const bool x_ok = tid < RST * QB && x_ul < RS && b_first + x_bl < q;
    const uint32_t x_off = (uint32_t)(x_ul * q + b_first + x_bl);

    auto issue_stage = [&](int s, int slot) {
        unsigned char *base = lds + slot * S::STAGE_BYTES;
        const int64_t kc0 = (int64_t)s * KA;
#pragma unroll
        for (int i = 0; i < S::A_CNT; ++i) {
            const uint32_t off = kc0 + a_col[i] < k ? a_off[i] + (uint32_t)(kc0 * 4) : OOB;
            lds_dma<S::A_W>(a_rsrc, base + (i * NW + wave) * 64 * S::A_W, off);
        }
        const int64_t u0 = (int64_t)s * RS;
        const int64_t rows_left = min<int64_t>(RS, w - u0);
        const __amdgpu_buffer_rsrc_t b_rsrc = make_rsrc(p.Bc + u0 * n, (uint32_t)(rows_left * n * 4));
#pragma unroll
        for (int i = 0; i < S::B_CNT; ++i)
            lds_dma<S::B_W>(b_rsrc, base + S::A_BYTES + (i * NW + wave) * 64 * S::B_W,
                            b_ok[i] ? b_off[i] : OOB);
        const __amdgpu_buffer_rsrc_t x_rsrc = make_rsrc(p.idx + u0 * q, (uint32_t)(rows_left * q));
        lds_dma<1>(x_rsrc, base + S::A_BYTES + S::B_BYTES + wave * 64 * 4, x_ok ? x_off : OOB);
    };

    f32x4 acc[NCG][NRC][BV];
#pragma unroll
    for (int cg = 0; cg < NCG; ++cg)
#pragma unroll
        for (int rc = 0; rc < NRC; ++rc)
#pragma unroll
            for (int s = 0; s < BV; ++s) acc[cg][rc][s] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int r = lane & 15, kq = lane >> 4;
    const int gps = KA / M;                         // windows per stage
    const int arow = wm * WM + r;                   // this lane's A row (chunk 0)
    const int swz = (arow >> 1) & 7;                // same for every chunk (16-row steps)

    auto compute_stage = [&](int slot) {
        const unsigned char *base = lds + slot * S::STAGE_BYTES;
        const unsigned char *Ab = base + arow * A_ROW_BYTES;
        const float *Bcol = reinterpret_cast<const float *>(base + S::A_BYTES) + wn * WN + BV * r;
        const int *Xs = reinterpret_cast<const int *>(base + S::A_BYTES + S::B_BYTES);
        int aoff[NQ][NCG];
#pragma unroll
        for (int qd = 0; qd < NQ; ++qd)
#pragma unroll
            for (int cg = 0; cg < NCG; ++cg) aoff[qd][cg] = Xs[(4 * qd + kq) * QB + blk[cg]];
#pragma unroll
        for (int qd = 0; qd < NQ; ++qd) {
            // window of this compressed row inside the stage; padding rows
            // (ul >= RS, zero in B_s) are clamped to the last window so that
            // they still address finite A_s data
            const int ul = 4 * qd + kq;
            const int window = min(ul / N, gps - 1) * M;
#pragma unroll
            for (int cg = 0; cg < NCG; ++cg) {
                const int c = window + min(aoff[qd][cg], M - 1);   // column of A_s gathered
                aoff[qd][cg] = ((((c >> 2) ^ swz) << 4) | ((c & 3) << 2));
            }
        }
        float a[2][NCG][NRC];
        bvec b[2][NCG];
        auto fetch = [&](int qd, int sl) {
#pragma unroll
            for (int cg = 0; cg < NCG; ++cg) {
#pragma unroll
                for (int rc = 0; rc < NRC; ++rc)
                    a[sl][cg][rc] = *reinterpret_cast<const float *>(Ab + aoff[qd][cg] + rc * 16 * A_ROW_BYTES);
                b[sl][cg] = *reinterpret_cast<const bvec *>(Bcol + (4 * qd + kq) * BN + cg * CG);
            }
        };
        fetch(0, 0);
#pragma unroll
        for (int qd = 0; qd < NQ; ++qd) {
            const int sl = qd & 1;
            if (qd + 1 < NQ) fetch(qd + 1, sl ^ 1);
            // keep the next quad's LDS reads ahead of this quad's MFMAs
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int cg = 0; cg < NCG; ++cg)
#pragma unroll
                for (int rc = 0; rc < NRC; ++rc)
#pragma unroll
                    for (int s = 0; s < BV; ++s)
                        acc[cg][rc][s] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                            a[sl][cg][rc], lane_of<BV>(b[sl][cg], s), acc[cg][rc][s], 0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    // ---- pipeline: P-1 stages in flight, one barrier per stage ----
#pragma unroll
    for (int j = 0; j < P - 1; ++j)
        if (j < nst) issue_stage(s_begin + j, j);
    for (int it = 0; it < nst; ++it) {
        wait_vm<LOADS, P - 2>(min(P - 2, nst - 1 - it));
        block_sync();
        if (it + P - 1 < nst) issue_stage(s_begin + it + P - 1, (it + P - 1) % P);
        compute_stage(it % P);
    }

    // ---- epilogue: lane l holds rows 4*(l/16)+v of each 16-row chunk and
    // columns BV*(l%16)+s of each column group ----
#pragma unroll
    for (int cg = 0; cg < NCG; ++cg) {
        const int64_t col = col0 + wn * WN + cg * CG + BV * r;
        if (col >= n) continue;
#pragma unroll
        for (int rc = 0; rc < NRC; ++rc)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int64_t row = row0 + wm * WM + rc * 16 + 4 * kq + v;
                if (row >= m) continue;
                float *dst = p.C + row * n + col;
                if (p.splits == 1) {
                    bvec out;
                    if constexpr (BV == 1) {
                        out = acc[cg][rc][0][v];
                    } else {
#pragma unroll
                        for (int s = 0; s < BV; ++s) out[s] = acc[cg][rc][s][v];
                    }
                    *reinterpret_cast<bvec *>(dst) = out;
                } else {
#pragma unroll
                    for (int s = 0; s < BV; ++s) unsafeAtomicAdd(dst + s, acc[cg][rc][s][v]);
                }
            }
    }
}

// Host-side launcher of one instantiation.
template <class T, int BV, int NQ>
hipError_t launch_tiled(const TiledArgs &a, hipStream_t stream)
{
    if constexpr (!Shape<T, BV, NQ>::FITS) {
        return hipErrorInvalidConfiguration;
    } else {
        const unsigned grid = (unsigned)a.tiles_m * (unsigned)a.tiles_n * (unsigned)a.splits;
        hipLaunchKernelGGL((nm_tiled_kernel<T, BV, NQ>), dim3(grid), dim3(T::NT), 0, stream, a);
        return hipGetLastError();
    }
}

// Dispatch over (BV, NQ) for one tile shape; NQ must be 1, 2, 3, 4 or 8.
template <class T>
hipError_t launch_tiled_any(int BV, int NQ, const TiledArgs &a, hipStream_t stream)
{
#define NMSPMM_NQ_CASES(bv)                                       \
    switch (NQ) {                                                 \
    case 1: return launch_tiled<T, bv, 1>(a, stream);             \
    case 2: return launch_tiled<T, bv, 2>(a, stream);             \
    case 3: return launch_tiled<T, bv, 3>(a, stream);             \
    case 4: return launch_tiled<T, bv, 4>(a, stream);             \
    case 8: return launch_tiled<T, bv, 8>(a, stream);             \
    default: return hipErrorInvalidValue;                         \
    }
    switch (BV) {
    case 1: NMSPMM_NQ_CASES(1)
    case 2: NMSPMM_NQ_CASES(2)
    case 4: NMSPMM_NQ_CASES(4)
    default: return hipErrorInvalidValue;
    }
#undef NMSPMM_NQ_CASES
}

template <class T>
constexpr bool tiled_fits(int BV, int NQ)
{
#define NMSPMM_FIT(bv, nq) (BV == bv && NQ == nq && Shape<T, bv, nq>::FITS)
    return NMSPMM_FIT(1, 1) || NMSPMM_FIT(1, 2) || NMSPMM_FIT(1, 3) || NMSPMM_FIT(1, 4) ||
           NMSPMM_FIT(1, 8) || NMSPMM_FIT(2, 1) || NMSPMM_FIT(2, 2) || NMSPMM_FIT(2, 3) ||
           NMSPMM_FIT(2, 4) || NMSPMM_FIT(2, 8) || NMSPMM_FIT(4, 1) || NMSPMM_FIT(4, 2) ||
           NMSPMM_FIT(4, 3) || NMSPMM_FIT(4, 4) || NMSPMM_FIT(4, 8);
#undef NMSPMM_FIT
}

}  // namespace nmspmm

#endif

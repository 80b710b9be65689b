// Tiled fp32-MFMA kernel for vector-wise N:M SpMM on gfx950 (device code,
// included by the per-shape instantiation units).
//
// One workgroup owns a BM x BN tile of C (and, with split-k, one slice of the
// k range).  It walks k in stages of KA columns of A (KA/M whole windows,
// RS = (KA/M)*N compressed rows, padded to RST = 4*NQ rows: MFMA K = 4).  KA
// grows as N/M shrinks so that a stage carries about sixteen compressed rows
// at every sparsity, the way the paper sizes k_s from the shared-memory budget
// and N/M (Sec. III-B.1, Eq. 5).  Each stage is brought into a ring of P LDS
// slots (the double buffer of Sec. III-C.2, deepened to P slots):
//   A_s : the BM x KA slab of A, row-major.  The whole slab is staged (the
//         non-packing load of Sec. III-C.1): with random per-block patterns
//         nearly every column is needed by some block of the tile.  Word c of
//         row i is stored at word position c ^ (i & 31), so that the sixteen
//         consecutive rows an MFMA gathers from one column fall in sixteen
//         different LDS banks.
//   B_s : the RST x BN slab of Bc, row-major (padding rows are zero).
//   X_s : the RST x (BN/V) offset bytes of D, one zero-extended dword each.
// All three are filled by buffer->LDS DMA (no register staging); each lane
// picks the global address whose data belongs at its fixed LDS position,
// which is how the swizzle is applied.  Out-of-range lanes (ragged m, n, k
// tails, padding rows) read zero.  Every wave issues the same number of DMA
// instructions per stage, so "a stage has landed" is a counted vmcnt wait
// followed by a barrier.
//
// Schedule (P >= 3): the barrier at the top of iteration s certifies that
// every wave is done with slot s-1 and that stage s has landed; the DMA of
// stage s+P-1 then refills slot s-1, so P-1 stages stay in flight behind the
// one being multiplied.  Inside a stage
// the offsets of all its quads are read once (the index prefetch of Sec.
// III-C.2) and the operands of quad q+1 are read while quad q is multiplied
// (the register double buffer of the same section).  With P == 2 the plain
// double buffer is used.
//
// Contraction: v_mfma_f32_16x16x4_f32 (fp32 in, fp32 accumulate).  Lane l
// supplies A[l%16][l/16] and B[l/16][l%16] and receives D[4*(l/16)+v][l%16]
// in element v.  The K index l/16 selects one of four consecutive compressed
// rows, each with its own gather offset; the 16 columns of one MFMA lie in a
// column group of CG = 16*BV columns inside one column block, so they share
// one gather.  A lanes read output row l%16 of a 16-row chunk; B lanes read
// columns BV*(l%16)+s, s < BV (BV MFMAs per A read).
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
constexpr int SWZ = 31;           // word swizzle mask of A_s rows (KA is a multiple of 32)

template <int BM_, int BN_, int WM_, int WN_>
struct TileCfg {
    static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_;
    static constexpr int NW = (BM / WM) * (BN / WN);
    static constexpr int NT = NW * 64;
    static constexpr int NRC = WM / 16;         // 16-row MFMA chunks per wave
    static_assert(WM % 16 == 0 && BM % WM == 0 && BN % WN == 0, "tile shape");
};

// Per-instantiation constants (tile x column-group width x stage shape).
template <class T, int BV, int KA, int NQ>
struct Shape {
    static constexpr int CG = 16 * BV;
    static constexpr int NCG = T::WN / CG;
    static constexpr int RST = 4 * NQ;                 // padded rows per stage
    static constexpr int QBMAX = T::BN / CG;           // column blocks per tile, at most
    static constexpr int A_ROW = KA * 4;               // bytes per A_s row
    static constexpr int A_BYTES = T::BM * A_ROW;
    static constexpr int B_BYTES = RST * T::BN * 4;
    static constexpr int X_BYTES = T::NT * 4;
    static constexpr int STAGE_BYTES = A_BYTES + B_BYTES + X_BYTES;
    // DMA instructions per wave per stage: A in dwords (word-level swizzle),
    // B in 16-byte pieces when the slab divides evenly, one byte of D per lane
    static constexpr int A_CNT = A_BYTES / (T::NT * 4);
    static constexpr int B_LANE = B_BYTES / T::NT;
    static constexpr int B_W = B_LANE % 16 == 0 ? 16 : 4;
    static constexpr int B_CNT = B_LANE / B_W;
    static constexpr int LOADS = A_CNT + B_CNT + 1;
    // ring depth: what LDS holds, at most 6, and few enough stages in flight
    // that a wait count (stages x LOADS) fits the 6-bit vmcnt
    static constexpr int P_LDS = LDS_CAPACITY / STAGE_BYTES;
    static constexpr int P_CNT = 2 + 63 / LOADS;
    static constexpr int P = P_LDS < P_CNT ? (P_LDS < 6 ? P_LDS : 6) : (P_CNT < 6 ? P_CNT : 6);
    static constexpr bool FITS = P >= 2 && KA % 32 == 0 && T::WN % CG == 0 &&
                                 RST * QBMAX <= T::NT && A_BYTES % (T::NT * 4) == 0 &&
                                 B_BYTES % T::NT == 0 && B_LANE % 4 == 0 && A_CNT >= 1 &&
                                 B_CNT >= 1 && (P - 2) * LOADS < 64;
};

struct TiledArgs {
    const float *A;
    const float *Bc;
    const uint8_t *idx;
    float *C;
    int64_t m, n, k;
    int N, M, V;
    int RS;          // real compressed rows per stage, (KA/M)*N
    int stages;      // ceil((k/M) / (KA/M))
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
// of the buffer land at dst + l*W.  (The width is spelled as a literal in
// each branch: the builtin needs an integer constant that is not
// template-dependent.)
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

// Wait until at most later_stages * LOADS DMA instructions of this wave are
// outstanding (s_waitcnt simm16 on gfx9: vmcnt[3:0] | expcnt[6:4] |
// lgkmcnt[11:8] | vmcnt[5:4] << 14; expcnt and lgkmcnt left at their maxima).
template <int LOADS, int MAXL>
__device__ __forceinline__ void wait_vm(int later_stages)
{
#define NMSPMM_VM(c) __builtin_amdgcn_s_waitcnt(((c) & 15) | (7 << 4) | (15 << 8) | (((c) >> 4) << 14))
    static_assert(MAXL <= 4 && MAXL * LOADS < 64, "ring depth");
    if constexpr (MAXL >= 4) { if (later_stages >= 4) { NMSPMM_VM(4 * LOADS); return; } }
    if constexpr (MAXL >= 3) { if (later_stages >= 3) { NMSPMM_VM(3 * LOADS); return; } }
    if constexpr (MAXL >= 2) { if (later_stages >= 2) { NMSPMM_VM(2 * LOADS); return; } }
    if constexpr (MAXL >= 1) { if (later_stages >= 1) { NMSPMM_VM(1 * LOADS); return; } }
    NMSPMM_VM(0);
#undef NMSPMM_VM
}

// Workgroup barrier without a memory fence: LDS visibility is established by
// the explicit vmcnt wait before it and the lgkmcnt(0) inside it; the empty
// asm statements keep the compiler from moving memory accesses across it.
__device__ __forceinline__ void block_sync()
{
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt((15) | (7 << 4) | (0 << 8) | (3 << 14));  // lgkmcnt(0)
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

template <class T, int BV, int KA, int NQ>
__global__ __launch_bounds__(T::NT) void nm_tiled_kernel(TiledArgs p)
{
    using S = Shape<T, BV, KA, NQ>;
    constexpr int BM = T::BM, BN = T::BN, WM = T::WM, WN = T::WN, NW = T::NW, NRC = T::NRC;
    constexpr int CG = S::CG, NCG = S::NCG, RST = S::RST, P = S::P, LOADS = S::LOADS;
    constexpr int A_ROW = S::A_ROW;
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
    // A DMA i of this wave fills word position (i*NW + wave)*64 + lane of
    // A_s: row a_row0 + i*AR (AR = NT/KA, a_row0 < AR) at in-row slot a_slot,
    // which holds column a_slot ^ (row & SWZ) = a_c0 ^ ((i*AR) & SWZ).
    constexpr int AR = T::NT / KA;
    static_assert(T::NT % KA == 0 && (AR & (AR - 1)) == 0, "A DMA rows");
    const int a_row0 = (wave * 64 + lane) / KA, a_slot = (wave * 64 + lane) % KA;
    const int a_c0 = a_slot ^ (a_row0 & SWZ);
    const uint32_t a_rowbase = (uint32_t)(a_row0 * k * 4);
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
        const bool full = kc0 + KA <= k;   // uniform; only a last, partial stage is not
#pragma unroll
        for (int i = 0; i < S::A_CNT; ++i) {
            const int col = a_c0 ^ ((i * AR) & SWZ);
            // the stage- and DMA-dependent part is made an opaque scalar so that
            // the per-lane offsets are formed here, not hoisted out of the loop
            const uint32_t su = __builtin_amdgcn_readfirstlane((uint32_t)((i * AR * k + kc0) * 4));
            const uint32_t off = a_rowbase + (uint32_t)col * 4u + su;
            lds_dma<4>(a_rsrc, base + (i * NW + wave) * 64 * 4, full || kc0 + col < k ? off : OOB);
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
    const int arow = wm * WM + r;                   // this lane's A row in chunk 0
    const int fsw = arow & SWZ;                     // its swizzle; chunk rc adds 16*rc

    // Gather offsets of one stage: byte offset inside the lane's A_s row for
    // even chunks (odd chunks sit 16 rows further, where the swizzle differs
    // in word bit 4, i.e. byte bit 6).
    int aoff[NQ][NCG];
    auto prep_offsets = [&](int slot) {
        const unsigned char *base = lds + slot * S::STAGE_BYTES;
        const int *Xs = reinterpret_cast<const int *>(base + S::A_BYTES + S::B_BYTES);
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
                aoff[qd][cg] = (c ^ fsw) * 4;
            }
        }
    };

    float a[2][NCG][NRC];
    bvec b[2][NCG];
    auto fetch = [&](int slot, int qd, int sl) {
        const unsigned char *base = lds + slot * S::STAGE_BYTES;
        const unsigned char *Ab = base + arow * A_ROW;
        const float *Bcol = reinterpret_cast<const float *>(base + S::A_BYTES) + wn * WN + BV * r;
#pragma unroll
        for (int cg = 0; cg < NCG; ++cg) {
#pragma unroll
            for (int rc = 0; rc < NRC; ++rc) {
                const int o = (rc & 1) ? (aoff[qd][cg] ^ 64) : aoff[qd][cg];
                a[sl][cg][rc] = *reinterpret_cast<const float *>(Ab + rc * 16 * A_ROW + o);
            }
            b[sl][cg] = *reinterpret_cast<const bvec *>(Bcol + (4 * qd + kq) * BN + cg * CG);
        }
    };
    auto mma = [&](int sl) {
#pragma unroll
        for (int cg = 0; cg < NCG; ++cg)
#pragma unroll
            for (int rc = 0; rc < NRC; ++rc)
#pragma unroll
                for (int s = 0; s < BV; ++s)
                    acc[cg][rc][s] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                        a[sl][cg][rc], lane_of<BV>(b[sl][cg], s), acc[cg][rc][s], 0, 0, 0);
    };

    if constexpr (P >= 3) {
        // ---- P-slot ring: P-1 stages in flight behind the one multiplied ----
#pragma unroll
        for (int j = 0; j < P - 1; ++j)
            if (j < nst) issue_stage(s_begin + j, j);
        if (nst > 0) {
            wait_vm<LOADS, P - 2>(min(nst - 1, P - 2));   // stage 0 landed
            block_sync();
        }
        for (int it = 0; it < nst; ++it) {
            const int slot = it % P;
            if (it > 0) {
                wait_vm<LOADS, P - 2>(min(nst - 1 - it, P - 2));  // stage it landed
                block_sync();
            }
            prep_offsets(slot);
            fetch(slot, 0, 0);
            if (it + P - 1 < nst) issue_stage(s_begin + it + P - 1, (it + P - 1) % P);
#pragma unroll
            for (int qd = 0; qd < NQ; ++qd) {
                const int sl = qd & 1;
                if (qd + 1 < NQ) fetch(slot, qd + 1, sl ^ 1);
                // keep the next LDS reads ahead of this quad's MFMAs
                __builtin_amdgcn_sched_barrier(0);
                mma(sl);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    } else {
        // ---- plain double buffer ----
        if (nst > 0) issue_stage(s_begin, 0);
        for (int it = 0; it < nst; ++it) {
            const int slot = it & 1;
            wait_vm<LOADS, 0>(0);
            block_sync();
            if (it + 1 < nst) issue_stage(s_begin + it + 1, slot ^ 1);
            prep_offsets(slot);
            fetch(slot, 0, 0);
#pragma unroll
            for (int qd = 0; qd < NQ; ++qd) {
                const int sl = qd & 1;
                if (qd + 1 < NQ) fetch(slot, qd + 1, sl ^ 1);
                __builtin_amdgcn_sched_barrier(0);
                mma(sl);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
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
template <class T, int BV, int KA, int NQ>
hipError_t launch_tiled(const TiledArgs &a, hipStream_t stream)
{
    if constexpr (!Shape<T, BV, KA, NQ>::FITS) {
        return hipErrorInvalidConfiguration;
    } else {
        const unsigned grid = (unsigned)a.tiles_m * (unsigned)a.tiles_n * (unsigned)a.splits;
        hipLaunchKernelGGL((nm_tiled_kernel<T, BV, KA, NQ>), dim3(grid), dim3(T::NT), 0, stream, a);
        return hipGetLastError();
    }
}

// The stage shapes instantiated: (KA, NQ), KA columns of A and 4*NQ padded
// compressed rows per stage.
#define NMSPMM_STAGE_SHAPES(X) \
    X(32, 1) X(32, 2) X(32, 3) X(32, 4) X(32, 8) X(64, 2) X(64, 4) X(128, 1) X(128, 2) X(128, 4)

template <class T, int BV>
hipError_t launch_tiled_bv(int KA, int NQ, const TiledArgs &a, hipStream_t stream)
{
#define NMSPMM_CASE(ka, nq) \
    if (KA == ka && NQ == nq) return launch_tiled<T, BV, ka, nq>(a, stream);
    NMSPMM_STAGE_SHAPES(NMSPMM_CASE)
#undef NMSPMM_CASE
    return hipErrorInvalidValue;
}

template <class T>
hipError_t launch_tiled_any(int BV, int KA, int NQ, const TiledArgs &a, hipStream_t stream)
{
    switch (BV) {
    case 1: return launch_tiled_bv<T, 1>(KA, NQ, a, stream);
    case 2: return launch_tiled_bv<T, 2>(KA, NQ, a, stream);
    case 4: return launch_tiled_bv<T, 4>(KA, NQ, a, stream);
    default: return hipErrorInvalidValue;
    }
}

template <class T, int BV>
constexpr bool tiled_fits_bv(int KA, int NQ)
{
#define NMSPMM_CASE(ka, nq) || (KA == ka && NQ == nq && Shape<T, BV, ka, nq>::FITS)
    return false NMSPMM_STAGE_SHAPES(NMSPMM_CASE);
#undef NMSPMM_CASE
}

template <class T>
constexpr bool tiled_fits(int BV, int KA, int NQ)
{
    return (BV == 1 && tiled_fits_bv<T, 1>(KA, NQ)) || (BV == 2 && tiled_fits_bv<T, 2>(KA, NQ)) ||
           (BV == 4 && tiled_fits_bv<T, 4>(KA, NQ));
}

}  // namespace nmspmm

#endif

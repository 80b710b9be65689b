// Tiled fp32-MFMA kernel for vector-wise N:M SpMM on gfx950 (device code,
// included by the per-shape instantiation units).
//
// One workgroup owns a BM x BN tile of C (and, with split-k, one slice of the
// k range).  It walks k in stages of KA columns of A (KA/M whole windows,
// RS = (KA/M)*N compressed rows, padded to RST = 4*NQ rows).  KA
// grows as N/M shrinks so that a stage carries about sixteen compressed rows
// at every sparsity, the way the paper sizes k_s from the shared-memory budget
// and N/M (Sec. III-B.1, Eq. 5).  Each stage is staged in one of two LDS
// slots (the double buffer of Sec. III-C.2):
//   A_s : the BM x KA slab of A, stored k-major (A_s[c][i], rows padded by 4
//         floats).  The whole slab is staged (the non-packing load of Sec.
//         III-C.1): with random per-block patterns nearly every column is
//         needed by some block of the tile.  k-major storage turns the N:M
//         gather of Eq. 1 into "pick LDS row c", and one 16-byte read gives
//         a lane RPL = 4 consecutive output rows of the gathered column.  It
//         goes global -> registers -> LDS: each thread loads a 4 x 4 block
//         (four 16-byte row pieces) and writes it transposed (four 16-byte
//         column pieces).
//   B_s : the RST x BN slab of Bc, row-major (padding rows are zero).
//   X_s : the RST x (BN/V) offset bytes of D, one zero-extended dword each.
// B_s and X_s are filled by buffer->LDS DMA.  All global reads go through
// buffer descriptors whose range makes ragged m / n / k tails and padding
// rows read zero.  The loads of stage s+1 are issued while stage s is
// multiplied; the A registers are written to the other slot after it; one
// barrier per stage.  (Deep stages of the tiles with few accumulators per
// lane keep a single A_s slot, written after a second barrier.)  Inside a stage the offsets of all MFMA K steps are read
// once (the index prefetch of Sec. III-C.2) and the operands of step j+1 are
// read while step j is multiplied (the register double buffer of the same
// section).
//
// Contraction: fp32 MFMA (fp32 in, fp32 accumulate), v_mfma_f32_16x16x4_f32
// or v_mfma_f32_32x32x2_f32 (MI = 16 or 32).  Lane l supplies A[l%MI][l/MI]
// and B[l/MI][l%MI]; the K index l/MI selects one of KG = 64/MI consecutive
// compressed rows, each with its own gather offset.  The MI columns of one
// MFMA lie in a column group of CG = MI*BV columns inside one column block,
// so they share one gather.  A lanes read output rows RPL*(l%MI)+t (t < RPL)
// of an MI*RPL-row chunk; B lanes read columns BV*(l%MI)+s (s < BV); one A
// read feeds RPL*BV MFMAs.
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

// MI selects the MFMA: 16 -> v_mfma_f32_16x16x4_f32 (K = 4 compressed rows,
// 16 lanes per K index), 32 -> v_mfma_f32_32x32x2_f32 (K = 2, 32 lanes per
// K index).  The 32 x 32 form issues half as many instructions for the same
// work and keeps the matrix pipe busier; it needs V to be a multiple of 32.
template <int BM_, int BN_, int WM_, int WN_, int MI_ = 16>
struct TileCfg {
    static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_, MI = MI_;
    static constexpr int NW = (BM / WM) * (BN / WN);
    static constexpr int NT = NW * 64;
    static constexpr int KG = 64 / MI;                 // K per MFMA (compressed rows)
    static constexpr int RPL = WM % (4 * MI) == 0 ? 4 : 1;  // output rows per lane read
    static constexpr int RCH = MI * RPL;               // rows per MFMA row chunk
    static constexpr int NRC = WM / RCH;
    static constexpr int AST = BM + 4;                 // floats per A_s row (k-major)
    static_assert(MI == 16 || MI == 32, "MFMA shape");
    static_assert(WM % MI == 0 && BM % WM == 0 && BN % WN == 0, "tile shape");
};

// Per-instantiation constants (tile x column-group width x stage shape).
template <class T, int BV, int KA, int NQ>
struct Shape {
    static constexpr int CG = T::MI * BV;
    static constexpr int NCG = T::WN / CG;
    static constexpr int RST = 4 * NQ;                 // padded rows per stage
    static constexpr int QBMAX = T::BN / CG;           // column blocks per tile, at most
    static constexpr int A_FLOATS = KA * T::AST;
    static constexpr int B_FLOATS = RST * T::BN;
    static constexpr int X_INTS = T::NT;
    // LDS: two slots of B_s and X_s (the loads of stage s+1 are in flight
    // while stage s is multiplied), and two slots of A_s where they fit.
    // Otherwise, for the tiles with at most 64 accumulators per lane, one
    // A_s slot: the A registers are the second buffer, and a barrier after
    // the last read of A_s lets them overwrite it.  This is what lets those
    // tiles take the deep stages of the sparsest levels: 128 x 256 at 4:32
    // and KA = 128 measured 11 % faster than at KA = 64 on MI355X.  The
    // 128-accumulator tiles have long enough stages at KA = 64; there the
    // extra barrier and the doubled A load burst measured slower.  (A
    // three-slot ring with loads two stages ahead measured within 1-3 % at
    // the cost of a second set of A staging registers, and spills on the
    // 128-accumulator tiles, so it is not used.)
    static constexpr int NSLOT = 2;
    static constexpr int A_BYTES = 4 * A_FLOATS;
    static constexpr int BX_BYTES = 4 * (B_FLOATS + X_INTS);
    static constexpr bool TWO_A = NSLOT * (A_BYTES + BX_BYTES) <= LDS_CAPACITY;
    static constexpr bool ONE_A_OK = T::BM * T::BN <= 64 * T::NT;
    static constexpr int A_SLOTS = TWO_A ? 2 : 1;
    static constexpr int SLOT_BYTES = A_BYTES + BX_BYTES;
    static constexpr int LDS_BYTES = A_SLOTS * A_BYTES + NSLOT * BX_BYTES;
    // A: chunks of A_RP rows x 32 columns, one per wave at a time, each
    // thread an (A_RP/8) x 4 block.  32-row chunks, or 16-row ones on the
    // 16-wave tiles where 32-row chunks would leave three quarters of the
    // waves without A work: the waves that load then load and store half as
    // much, and they set the stage's pace.  Measured on MI355X (per-launch
    // events): 2048 x 4096 x 4096 at 16:32 on 128 x 256 tiles (KA = 32)
    // 317.4 -> 306.8 us; where 32-row chunks already kept half the waves busy
    // (4096^3 at 16:32 and 8:32, 2048 x 4096 x 4096 at 8:32) it measured
    // within -0.3 / +0.5 %.
    static constexpr int A_CH32 = ((T::BM + 31) / 32) * (KA / 32);
    static constexpr int A_RP = (T::NT >= 1024 && (4 * A_CH32 <= T::NW || (NQ == 8 && A_CH32 <= T::NW))) ? 16 : 32;
    static constexpr int A_RL = A_RP / 8;               // rows per thread
    static constexpr int A_CHUNKS = ((T::BM + A_RP - 1) / A_RP) * (KA / 32);
    static constexpr int ACH = (A_CHUNKS + T::NW - 1) / T::NW;
    // B DMA: 16-byte pieces when the slab divides evenly, else dwords
    static constexpr int B_LANE = B_FLOATS * 4 / T::NT;
    static constexpr int B_W = B_LANE % 16 == 0 ? 16 : 4;
    static constexpr int B_CNT = B_LANE / B_W;
    // 16-wave tiles run four waves per SIMD, 128 VGPRs each: one A staging
    // chunk per wave and at most four quads per stage (more spill)
    static constexpr bool REGS_OK = T::NT < 1024 || ((NQ <= 4 || (NQ == 8 && A_RP == 16)) && ACH == 1);
    static constexpr bool FITS = (TWO_A || ONE_A_OK) && REGS_OK && LDS_BYTES <= LDS_CAPACITY &&
                                 KA % 32 == 0 &&
                                 T::WN % CG == 0 && RST * QBMAX <= T::NT &&
                                 (B_FLOATS * 4) % T::NT == 0 && B_LANE % 4 == 0 && B_CNT >= 1;
};

// Output epilogue act(alpha * c + bias[j]) (see nmspmm_run_ex).
struct Epilogue {
    float alpha;
    const float *bias;   // n values or null
    int act;             // nmspmm_act_t
};

__device__ __forceinline__ float apply_epilogue(const Epilogue &e, float v, int64_t col)
{
    v *= e.alpha;
    if (e.bias) v += e.bias[col];
    if (e.act == 1) {
        v = fmaxf(v, 0.f);
    } else if (e.act == 2) {
        v = 0.5f * v * (1.f + erff(v * 0.70710678118654752f));
    }
    return v;
}

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
    Epilogue epi;    // applied by the stores when splits == 1
    int64_t col_begin = 0;   // first column of the tile grid (a multiple of BN and of V)
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

// 64-bit integer min / max.  (HIP's device min / max templates resolve a call
// whose two arguments differ in type, e.g. min<int64_t>(x, 4), to an overload
// that computes in double.)
__device__ __forceinline__ int64_t min64(int64_t a, int64_t b) { return a < b ? a : b; }
__device__ __forceinline__ int64_t max64(int64_t a, int64_t b) { return a > b ? a : b; }

// Debug build switch (off in the product library): with NMSPMM_POISON_LDS=1
// every buffer->LDS DMA first fills its own destination with NaN (offset
// bytes: a NaN bit pattern, which the readers clamp to the last offset of
// the window, a wrong but in-bounds column), waits for those stores, then
// issues the DMA; the tiled kernel also fills each A_s slot with NaN as soon
// as it is free.  A reader that runs ahead of a missing wait or barrier then
// reads NaN or a wrong column instead of stale data that may happen to be
// right, and the exact-result tests fail.
#ifndef NMSPMM_POISON_LDS
#define NMSPMM_POISON_LDS 0
#endif

// One buffer->LDS DMA instruction: lane l's W bytes from byte offset `off`
// of the buffer land at dst + l*W (W = 1: a zero-extended dword at dst +
// l*4).  (The width is spelled as a literal in each branch: the builtin needs
// an integer constant that is not template-dependent.)
template <int W>
__device__ __forceinline__ void lds_dma(__amdgpu_buffer_rsrc_t rsrc, void *dst, uint32_t off)
{
    static_assert(W == 1 || W == 4 || W == 16, "DMA width");
    if constexpr (NMSPMM_POISON_LDS) {
        const int l = (int)__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
        const float nan = __builtin_nanf("");
        if constexpr (W == 16)
            *reinterpret_cast<f32x4 *>(static_cast<unsigned char *>(dst) + 16 * l) = f32x4{nan, nan, nan, nan};
        else
            *reinterpret_cast<float *>(static_cast<unsigned char *>(dst) + 4 * l) = nan;
        __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14));  // lgkmcnt(0)
    }
    if constexpr (W == 16)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void *)dst, 16, (int)off, 0, 0, 0);
    else if constexpr (W == 4)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void *)dst, 4, (int)off, 0, 0, 0);
    else
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void *)dst, 1, (int)off, 0, 0, 0);
}

// Workgroup barrier after this wave's LDS accesses have completed; its
// global loads and DMA stay in flight.
__device__ __forceinline__ void lds_sync()
{
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14));  // lgkmcnt(0)
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// Workgroup barrier after this wave's outstanding global loads and DMA have
// completed (vmcnt(0)) and its LDS accesses have too (lgkmcnt(0)).  No memory
// fence beyond that is needed; the empty asm statements keep the compiler
// from moving memory accesses across it.
__device__ __forceinline__ void stage_sync()
{
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(0 | (7 << 4) | (0 << 8) | (0 << 14));  // vmcnt(0) lgkmcnt(0)
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

template <class T, int BV, int KA, int NQ>
__global__ __launch_bounds__(T::NT) void nm_tiled_kernel(TiledArgs p)
{
    using S = Shape<T, BV, KA, NQ>;
    constexpr int BM = T::BM, BN = T::BN, WM = T::WM, WN = T::WN, NW = T::NW;
    constexpr int RPL = T::RPL, RCH = T::RCH, NRC = T::NRC, AST = T::AST;
    constexpr int CG = S::CG, NCG = S::NCG, RST = S::RST, ACH = S::ACH;
    typedef typename vec_of<BV>::type bvec;
    typedef typename vec_of<RPL>::type avec;

    __shared__ __align__(16) unsigned char lds[S::LDS_BYTES];
    // A_s of a slot, and B_s followed by X_s of a slot.  Two A slots: slot i
    // is A_s, B_s, X_s at i * SLOT_BYTES, so that slot 0's B_s stays within
    // the 16-bit offsets of LDS instructions.  One A slot: A_s, then the two
    // B_s / X_s slots.
    auto a_area = [&](int slot) -> unsigned char * {
        if constexpr (S::TWO_A) return lds + slot * S::SLOT_BYTES;
        else return lds;
    };
    auto bx_area = [&](int slot) -> unsigned char * {
        if constexpr (S::TWO_A) return lds + slot * S::SLOT_BYTES + S::A_BYTES;
        else return lds + S::A_BYTES + slot * S::BX_BYTES;
    };

    const int tid = threadIdx.x, lane = tid & 63;
    // uniform across the wave.  Saying so lets the 32x32 tiles keep their
    // address math in scalar registers (measured 1-2 % faster); the 16x16
    // tiles measured slightly slower with it.
    const int wave = T::MI == 32 ? __builtin_amdgcn_readfirstlane(tid >> 6) : tid >> 6;
    int tm, tn, split;
    map_tile(blockIdx.x, gridDim.x, p.tiles_m, p.tiles_n, tm, tn, split);
    const int64_t row0 = (int64_t)tm * BM, col0 = p.col_begin + (int64_t)tn * BN;
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

    // ---- A: global -> registers (A_RL x 4 blocks) -> LDS, k-major ----
    // In an A_RP x 32 chunk, lane l owns rows A_RL*(l%8)+t (t < A_RL) and
    // columns 4*(l/8)..+3: each load instruction covers 8 rows x 128 bytes.
    constexpr int A_RP = S::A_RP, A_RL = S::A_RL, A_PC = (BM + A_RP - 1) / A_RP;
    typedef typename vec_of<A_RL>::type arvec;
    const int r8 = lane & 7, c8 = lane >> 3;
    const int rows_valid = (int)min64(BM, m - row0);
    const __amdgpu_buffer_rsrc_t a_rsrc =
        make_rsrc(p.A + row0 * k, (uint32_t)((int64_t)rows_valid * k * 4));
    f32x4 ra[ACH][A_RL];
    // `valid` false: the loads are still issued (so that every stage issues
    // the same memory instructions) but read zeros
    auto load_a = [&](int s, bool valid) {
        const int64_t kc0 = (int64_t)s * KA;
#pragma unroll
        for (int ch = 0; ch < ACH; ++ch) {
            const int chunk = wave + ch * NW;
            const int rbase = (chunk % A_PC) * A_RP, cbase = (chunk / A_PC) * 32;
            const int64_t kcol = kc0 + cbase + 4 * c8;
#pragma unroll
            for (int t = 0; t < A_RL; ++t) {
                const int r = rbase + A_RL * r8 + t;
                const bool ok = valid && chunk < S::A_CHUNKS && r < BM && kcol < k;
                const uint32_t off = ok ? (uint32_t)((r * k + kcol) * 4) : OOB;
                // the buffer load returns raw dwords; reinterpret them as floats
                ra[ch][t] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(a_rsrc, (int)off, 0, 0));
            }
        }
    };
    auto store_a = [&](int slot) {
        float *As = reinterpret_cast<float *>(a_area(slot));
#pragma unroll
        for (int ch = 0; ch < ACH; ++ch) {
            const int chunk = wave + ch * NW;
            const int rbase = (chunk % A_PC) * A_RP, cbase = (chunk / A_PC) * 32;
            if (chunk < S::A_CHUNKS && rbase + A_RL * r8 < BM) {
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    arvec v;
                    if constexpr (A_RL == 4)
                        v = arvec{ra[ch][0][c], ra[ch][1][c], ra[ch][2][c], ra[ch][3][c]};
                    else
                        v = arvec{ra[ch][0][c], ra[ch][1][c]};
                    *reinterpret_cast<arvec *>(As + (cbase + 4 * c8 + c) * AST + rbase + A_RL * r8) = v;
                }
            }
        }
    };

    // ---- B and D offsets: buffer -> LDS DMA ----
    uint32_t b_off[S::B_CNT];
    bool b_ok[S::B_CNT];
#pragma unroll
    for (int i = 0; i < S::B_CNT; ++i) {
        const int pos = ((i * NW + wave) * 64 + lane) * S::B_W;   // byte position in B_s
        const int ul = pos / (BN * 4), col = (pos % (BN * 4)) / 4;
        b_ok[i] = col0 + col < n;
        b_off[i] = (uint32_t)(((int64_t)ul * n + col0 + col) * 4);
    }
    // X_s holds, per column block of the tile, the stage's offsets in the
    // order a lane reads them: entry blk*RST + kq*NKS + ks is compressed row
    // KG*ks + kq, so that one lane's NKS offsets are contiguous
    constexpr int NKS_X = RST / (64 / T::MI);
    const int x_bl = tid / RST, x_kq = (tid % RST) / NKS_X, x_ks = tid % NKS_X;
    const int x_ul = (64 / T::MI) * x_ks + x_kq;
    const bool x_ok = tid < RST * QB && x_ul < RS && b_first + x_bl < q;
    const uint32_t x_off = (uint32_t)(x_ul * q + b_first + x_bl);
    auto dma_bx = [&](int s, int slot, bool valid) {
        unsigned char *bs = bx_area(slot);
        const int64_t u0 = (int64_t)s * RS;
        const int64_t rows_left = valid ? max64(0, min64(RS, w - u0)) : 0;
        const __amdgpu_buffer_rsrc_t b_rsrc = make_rsrc(p.Bc + u0 * n, (uint32_t)(rows_left * n * 4));
#pragma unroll
        for (int i = 0; i < S::B_CNT; ++i)
            lds_dma<S::B_W>(b_rsrc, bs + (i * NW + wave) * 64 * S::B_W, b_ok[i] ? b_off[i] : OOB);
        const __amdgpu_buffer_rsrc_t x_rsrc = make_rsrc(p.idx + u0 * q, (uint32_t)(rows_left * q));
        lds_dma<1>(x_rsrc, bs + 4 * S::B_FLOATS + wave * 64 * 4, x_ok ? x_off : OOB);
    };

    constexpr int MI = T::MI, KG = T::KG;
    constexpr int NKS = RST / KG;                   // MFMA K steps per stage
    constexpr int NACC = MI * MI / 64;              // accumulator floats per lane per MFMA
    typedef float accv __attribute__((ext_vector_type(NACC)));
    accv acc[NCG][NRC][RPL][BV];
#pragma unroll
    for (int cg = 0; cg < NCG; ++cg)
#pragma unroll
        for (int rc = 0; rc < NRC; ++rc)
#pragma unroll
            for (int t = 0; t < RPL; ++t)
#pragma unroll
                for (int s = 0; s < BV; ++s)
#pragma unroll
                    for (int e = 0; e < NACC; ++e) acc[cg][rc][t][s][e] = 0.f;

    const int r = lane % MI, kq = lane / MI;        // lane's row/column index, K index
    const int gps = KA / M;                         // windows per stage

    // Gather offsets of one stage: byte offset of the A_s row (column of A)
    // each of this lane's compressed rows reads, per column group.
    int aoff[NKS][NCG];
    auto prep_offsets = [&](int slot) {
        const int *Xs = reinterpret_cast<const int *>(bx_area(slot) + 4 * S::B_FLOATS);
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks)
#pragma unroll
            for (int cg = 0; cg < NCG; ++cg) aoff[ks][cg] = Xs[blk[cg] * RST + kq * NKS + ks];
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) {
            // window of this compressed row inside the stage; padding rows
            // (ul >= RS, zero in B_s) are clamped to the last window so that
            // they still address finite A_s data
            const int ul = KG * ks + kq;
            const int window = min(ul / N, gps - 1) * M;
#pragma unroll
            for (int cg = 0; cg < NCG; ++cg)
                aoff[ks][cg] = (window + min(aoff[ks][cg], M - 1)) * (AST * 4);
        }
    };

    avec a[2][NCG][NRC];
    bvec b[2][NCG];
    auto fetch = [&](int slot, int ks, int sl) {
        const unsigned char *base = a_area(slot);
        const unsigned char *Ab = base + (wm * WM + RPL * r) * 4;
        const float *Bcol = reinterpret_cast<const float *>(S::TWO_A ? base + S::A_BYTES : bx_area(slot)) +
                            wn * WN + BV * r;
#pragma unroll
        for (int cg = 0; cg < NCG; ++cg) {
#pragma unroll
            for (int rc = 0; rc < NRC; ++rc)
                a[sl][cg][rc] = *reinterpret_cast<const avec *>(Ab + aoff[ks][cg] + rc * RCH * 4);
            b[sl][cg] = *reinterpret_cast<const bvec *>(Bcol + (KG * ks + kq) * BN + cg * CG);
        }
    };
    auto mma = [&](int sl) {
#pragma unroll
        for (int cg = 0; cg < NCG; ++cg)
#pragma unroll
            for (int rc = 0; rc < NRC; ++rc)
#pragma unroll
                for (int t = 0; t < RPL; ++t)
#pragma unroll
                    for (int s = 0; s < BV; ++s) {
                        if constexpr (MI == 16)
                            acc[cg][rc][t][s] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                                lane_of<RPL>(a[sl][cg][rc], t), lane_of<BV>(b[sl][cg], s),
                                acc[cg][rc][t][s], 0, 0, 0);
                        else
                            acc[cg][rc][t][s] = __builtin_amdgcn_mfma_f32_32x32x2f32(
                                lane_of<RPL>(a[sl][cg][rc], t), lane_of<BV>(b[sl][cg], s),
                                acc[cg][rc][t][s], 0, 0, 0);
                    }
    };

    // ---- double-buffered stages, one barrier each ----
    // Stage i lives in LDS slot i % 2.  Its loads are issued while stage i-1
    // is multiplied, its A loads after that stage's first MFMA K step and its
    // DMA after the second: a wave whose memory instructions stall at issue
    // then still has MFMAs in the pipe (issuing them before the first MFMA
    // cost 5-12 % on MI355X; splitting them over two K steps measured 4096^3
    // at 16:32 530.7 -> 525.2 us, 2048 x 11008 x 4096 at 8:32 440.6 -> 434.1).  Its A
    // registers go to LDS at the end of stage i-1, and the barrier that
    // follows waits for them and for its DMA.  Every stage issues its loads
    // and its A store unconditionally (loads past the last stage read zeros),
    // so the compiler's wait counts see one straight-line pattern.
    if (nst > 0) {
        load_a(s_begin, true);
        dma_bx(s_begin, 0, true);
        store_a(0);
        stage_sync();
    }
    for (int it = 0; it < nst; ++it) {
        const int cur = it & 1;
        const bool next = it + 1 < nst;
        if constexpr (NMSPMM_POISON_LDS && S::TWO_A) {
            // the other A_s slot is free (every wave passed the barrier after
            // its last read): NaN in the places this wave's store will fill
            const float nan = __builtin_nanf("");
#pragma unroll
            for (int ch = 0; ch < ACH; ++ch)
#pragma unroll
                for (int t = 0; t < A_RL; ++t) ra[ch][t] = f32x4{nan, nan, nan, nan};
            store_a(cur ^ 1);
        }
        prep_offsets(cur);
        fetch(cur, 0, 0);
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) {
            const int sl = ks & 1;
            if (ks + 1 < NKS) fetch(cur, ks + 1, sl ^ 1);
            // keep the next LDS reads ahead of this step's MFMAs
            __builtin_amdgcn_sched_barrier(0);
            mma(sl);
            __builtin_amdgcn_sched_barrier(0);
            // the next stage's A loads after this stage's first K step, its
            // DMA after the second: a wave's memory instructions then stall
            // its issue for two shorter spells
            if (ks == 0) load_a(s_begin + it + 1, next);
            if (ks == (NKS > 1 ? 1 : 0)) dma_bx(s_begin + it + 1, cur ^ 1, next);
        }
        // one A_s slot: every wave must be done reading it
        if constexpr (!S::TWO_A) lds_sync();
        store_a(cur ^ 1);
        stage_sync();
    }

    // ---- epilogue.  16x16x4: element e of lane l is row 4*(l/16)+e of the
    // MFMA tile; 32x32x2: row 8*(e/4) + 4*(l/32) + e%4.  The MFMA tile row i
    // is output row RPL*i+t of its row chunk; its column is BV*(l%MI)+s of
    // the column group. ----
#pragma unroll
    for (int cg = 0; cg < NCG; ++cg) {
        const int64_t col = col0 + wn * WN + cg * CG + BV * r;
        if (col >= n) continue;
#pragma unroll
        for (int rc = 0; rc < NRC; ++rc)
#pragma unroll
            for (int e = 0; e < NACC; ++e)
#pragma unroll
                for (int t = 0; t < RPL; ++t) {
                    const int i = MI == 16 ? 4 * kq + e : 8 * (e / 4) + 4 * kq + (e % 4);
                    const int64_t row = row0 + wm * WM + rc * RCH + RPL * i + t;
                    if (row >= m) continue;
                    float *dst = p.C + row * n + col;
                    if (p.splits == 1) {
                        bvec out;
                        if constexpr (BV == 1) {
                            out = apply_epilogue(p.epi, acc[cg][rc][t][0][e], col);
                        } else {
#pragma unroll
                            for (int s = 0; s < BV; ++s)
                                out[s] = apply_epilogue(p.epi, acc[cg][rc][t][s][e], col + s);
                        }
                        *reinterpret_cast<bvec *>(dst) = out;
                    } else {
#pragma unroll
                        for (int s = 0; s < BV; ++s) unsafeAtomicAdd(dst + s, acc[cg][rc][t][s][e]);
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
    X(32, 1) X(32, 2) X(32, 3) X(32, 4) X(32, 8) X(64, 2) X(64, 4) X(64, 8) X(128, 1) X(128, 2) X(128, 4)

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

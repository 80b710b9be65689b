// Device half of the C ABI: the general kernel, the split-k zero fill and
// the dispatch behind nmspmm_run (the tiled MFMA kernel lives in
// nmspmm_tiled.h, instantiated per tile shape in nmspmm_tiled_*.hip; the
// streaming kernels for short products in nmspmm_skinny.hip and
// nmspmm_stream.hip; the direct-gather kernel of the workspace entry point in
// nmspmm_gather.hip).
//
// Notation as in the public header: A m x k, Bc w x n, idx w x q (uint8),
// C m x n; w = (k/M)*N, q = n/V; compressed row u belongs to window u/N.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>

#include "nmspmm.h"
#include "nmspmm_gather.h"
#include "nmspmm_internal.h"
#include "nmspmm_rowgather.h"
#include "nmspmm_skinny.h"
#include "nmspmm_stream.h"
#include "nmspmm_tiled.h"
#include "nmspmm_tiles.h"

namespace nmspmm {
namespace {

// ---------------------------------------------------------------------------
// General kernel: any legal (N, M, V) and any alignment.  One thread per
// output column, GEN_ROWS rows per pass; every term of Eq. 1 is read straight
// from global memory (the caches serve the reuse).  It covers the shapes the
// tiled kernel does not (V not a multiple of 16, M not dividing 32, k not a
// multiple of 4, unaligned buffers); it is not tuned.
// ---------------------------------------------------------------------------
constexpr int GEN_COLS = 256;
constexpr int GEN_ROWS = 8;

__global__ __launch_bounds__(GEN_COLS) void nm_general_kernel(
    const float *__restrict__ A, const float *__restrict__ Bc, const uint8_t *__restrict__ idx,
    float *__restrict__ C, int64_t m, int64_t n, int64_t k, int N, int M, int V, Epilogue epi)
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
            if (i0 + r < m) C[(i0 + r) * n + j] = apply_epilogue(epi, acc[r], j);
    }
}

// The epilogue of a split-k launch, once the atomic sums are complete: one
// pass over C.
__global__ __launch_bounds__(256) void nm_epilogue_kernel(float *__restrict__ C, int64_t count,
                                                           int64_t n, Epilogue epi)
{
    const int64_t stride = (int64_t)gridDim.x * 256;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < count; i += stride)
        C[i] = apply_epilogue(epi, C[i], i % n);
}

// Zero C before a split-k launch accumulates into it (a kernel, not a
// memset, so the sequence can be captured into a graph).
__global__ __launch_bounds__(256) void nm_zero_kernel(float *__restrict__ C, int64_t count)
{
    const int64_t stride = (int64_t)gridDim.x * 256;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < count; i += stride) C[i] = 0.f;
}

// The same with 16-byte stores, for a 16-byte aligned C (count4 = count / 4;
// the last count % 4 floats are cleared by the first threads).
__global__ __launch_bounds__(256) void nm_zero4_kernel(float *__restrict__ C, int64_t count)
{
    const int64_t stride = (int64_t)gridDim.x * 256, count4 = count / 4;
    const int64_t first = (int64_t)blockIdx.x * 256 + threadIdx.x;
    float4 *C4 = reinterpret_cast<float4 *>(C);
    for (int64_t i = first; i < count4; i += stride) C4[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (first < count - 4 * count4) C[4 * count4 + first] = 0.f;
}

// The second half of a split-k launch through a workspace: one thread per
// output, the partial tiles of its output tile (tile-major, splits
// consecutive, row-major ROWS x COLS each) summed in split order, then the
// epilogue.  Consecutive threads take consecutive columns of a tile row.
__global__ __launch_bounds__(256) void nm_splitk_reduce_kernel(const float *__restrict__ ws,
                                                               float *__restrict__ C, int64_t m, int64_t n,
                                                               int rows, int cols, int tiles_n, int splits,
                                                               Epilogue epi)
{
    const int64_t count = m * n;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < count; i += (int64_t)gridDim.x * 256) {
        const int64_t row = i / n, col = i - row * n;
        const int64_t tile = (row / rows) * tiles_n + col / cols;
        const int64_t e = (row % rows) * cols + col % cols;
        const int64_t tsz = (int64_t)rows * cols;
        const float *p = ws + tile * splits * tsz + e;
        float sum = p[0];
        for (int s = 1; s < splits; ++s) sum += p[s * tsz];
        C[i] = apply_epilogue(epi, sum, col);
    }
}

// ---------------------------------------------------------------------------
// Dispatch
// ---------------------------------------------------------------------------
struct TileInfo {
    const char *name;
    int BM, BN, MI, waves;
    hipError_t (*launch)(int, int, int, const TiledArgs &, hipStream_t);
    bool (*fits)(int, int, int);
};

const TileInfo TILES[] = {
    {"256x256", 256, 256, 16, 8, launch_tiled_256x256, tiled_fits_256x256},
    {"128x512", 128, 512, 16, 8, launch_tiled_128x512, tiled_fits_128x512},
    {"128x128", 128, 128, 16, 4, launch_tiled_128x128, tiled_fits_128x128},
    {"64x512", 64, 512, 16, 8, launch_tiled_64x512, tiled_fits_64x512},
    {"16x512", 16, 512, 16, 8, launch_tiled_16x512, tiled_fits_16x512},
    {"256x256m32", 256, 256, 32, 8, launch_tiled_256x256m32, tiled_fits_256x256m32},
    {"128x512m32", 128, 512, 32, 8, launch_tiled_128x512m32, tiled_fits_128x512m32},
    {"128x128m32", 128, 128, 32, 2, launch_tiled_128x128m32, tiled_fits_128x128m32},
    {"64x512m32", 64, 512, 32, 8, launch_tiled_64x512m32, tiled_fits_64x512m32},
    {"128x256", 128, 256, 16, 8, launch_tiled_128x256, tiled_fits_128x256},
    {"256x128", 256, 128, 16, 8, launch_tiled_256x128, tiled_fits_256x128},
    {"128x256m32", 128, 256, 32, 8, launch_tiled_128x256m32, tiled_fits_128x256m32},
    {"64x1024m32", 64, 1024, 32, 8, launch_tiled_64x1024m32, tiled_fits_64x1024m32},
    {"256x256m32w16", 256, 256, 32, 16, launch_tiled_256x256m32w16, tiled_fits_256x256m32w16},
    {"128x512m32w16", 128, 512, 32, 16, launch_tiled_128x512m32w16, tiled_fits_128x512m32w16},
    {"128x256m32w16", 128, 256, 32, 16, launch_tiled_128x256m32w16, tiled_fits_128x256m32w16},
};
constexpr int NTILES = sizeof(TILES) / sizeof(TILES[0]);

const TileInfo *tile_by_name(const char *name)
{
    for (int i = 0; i < NTILES; ++i)
        if (std::strcmp(TILES[i].name, name) == 0) return &TILES[i];
    return nullptr;
}

enum class Kind { None, General, Tiled, Skinny, Stream, Gather, RowGather };

struct Plan {
    Kind kind = Kind::None;
    const TileInfo *tile = nullptr;
    int BV = 0, KA = 0, NQ = 0, RS = 0, stages = 0, splits = 1, tiles_m = 0, tiles_n = 0;
    int QPW = 0, COLS = 0, CW = 0, RT = 1;   // streaming kernels only
    int CPW = 0, RB = 0, SW = 0;             // pipelined streaming kernel only
    int CT = 0, NW = 0, D = 0;               // direct-gather kernel only
    int H = 1;                               // its row halves
    int64_t ws_bytes = 0;
    // tiled kernel over two column regions (split-k off): columns [0,
    // col_split) with `tile` as above, then [col_split, n) with tile2
    const TileInfo *tile2 = nullptr;
    int BV2 = 0, KA2 = 0, NQ2 = 0, stages2 = 0, tiles_n2 = 0;
    int64_t col_split = 0;
};

bool aligned(const void *p, int bytes) { return (reinterpret_cast<uintptr_t>(p) % bytes) == 0; }

// Workspace of a split-k launch of the pipelined streaming kernel (0 when
// the plan does not take one): tiles * splits partial tiles.  Measured on
// MI355X against atomic adds into a zeroed C: 64 x 8192 x 8192 at 4:32
// 27.6 -> 25.0 us, 128 x 8192 x 8192 40.5 -> 39.0.  The register-operand
// streaming kernel keeps the atomics: its 16-row tiles add little, and the
// reduction pass cost more than they did (16 x 8192 x 8192 15.0 -> 15.8 us).
int64_t plan_ws_bytes(const Plan &p)
{
    if (p.kind == Kind::Gather) return p.ws_bytes;
    if (p.splits <= 1 || p.kind != Kind::Stream) return 0;
    const int64_t tiles = (int64_t)p.tiles_m * p.tiles_n;
    return tiles * p.splits * stream_rows(p.RT) * p.COLS * 4;
}

// Quads per stage actually instantiated for a stage depth of KA columns of A
// (the smallest that holds RS compressed rows), 0 if none.
int stage_nq(int KA, int RS)
{
    static const int shapes[][2] = {{32, 1}, {32, 2}, {32, 3}, {32, 4}, {32, 8},
                                    {64, 2}, {64, 4}, {64, 8}, {128, 1}, {128, 2}, {128, 4}};
    int best = 0;
    for (const auto &sh : shapes) {
        // (64, 8) only for whole stages of 32 rows (the deep stages of the
        // 16-wave tiles), never as padding
        if (sh[0] == 64 && sh[1] == 8 && RS != 32) continue;
        if (sh[0] == KA && 4 * sh[1] >= RS && (best == 0 || sh[1] < best)) best = sh[1];
    }
    return best;
}

// Column-group width of one MFMA read of B (columns per lane) for an MFMA of
// MI columns: the widest of 4 / 2 / 1 whose group MI*BV divides V; 0 if none.
int bv_for(int MI, int V)
{
    for (int bv : {4, 2, 1})
        if (V % (MI * bv) == 0) return bv;
    return 0;
}

bool tile_ok(const TileInfo &t, int BV, int KA, int NQ, int64_t k, int V)
{
    if (!(t.BN % V == 0 || V % t.BN == 0)) return false;
    if (!t.fits(BV, KA, NQ)) return false;
    return (int64_t)t.BM * k * 4 < (int64_t(1) << 31);
}

// Accumulator floats per lane: tiles with at most 64 fit two workgroups per
// CU when their stage is shallow, the others one.
int acc_per_lane(const TileInfo &t) { return t.BM * t.BN / (64 * t.waves); }

// 8-wave tiles with at most 64 accumulators per lane run two workgroups per
// CU; 16-wave tiles (four waves per SIMD) run one.
bool two_per_cu(const TileInfo &t) { return t.waves <= 8 && acc_per_lane(t) <= 64; }

// Fraction of the workgroup slots a tile grid keeps busy over its waves of
// workgroups (the last wave is usually partial), with slots = CUs x
// workgroups per CU.
double occupancy_of_grid(const TileInfo &t, int64_t m, int64_t n)
{
    const int64_t tiles = ((m + t.BM - 1) / t.BM) * ((n + t.BN - 1) / t.BN);
    const int64_t slots = 256 * (two_per_cu(t) ? 2 : 1);
    const int64_t rounds = (tiles + slots - 1) / slots;
    return (double)tiles / (double)(rounds * slots);
}

// Tile-shape preference by problem size, from sweeps on MI355X:
//  * m <= 128 (when the streaming kernel does not apply): 16- and 64-row
//    tiles with split-k, which keep enough workgroups in flight to stream Bc;
//  * m or n below 1024: the 128 x 256 tile with 32 x 32 MFMAs, else the
//    128 x 128 tile (enough tiles to fill the chip, with split-k);
//  * otherwise, at N/M <= 1/2 with V a multiple of 32, a 16-wave tile when
//    its grid fills the chip in one round (at most 256 tiles, at least three
//    quarters of the CUs busy): 128 x 512, else (at N/M = 1/2) 256 x 256,
//    else 128 x 256.  Four waves per SIMD hide the A loads of one wave behind
//    the MFMAs of the others (4096^3 at 16:32 566 -> 543 us, at 4:32 184 ->
//    163 us); on grids of several rounds (2048 x 11008) and on split-k grids
//    the 8-wave tiles measured faster.  At N/M = 1/2 the 128 x 512 tile,
//    whose stage offsets come in 16-byte reads, measured ahead of 256 x 256
//    (per-launch events, 4096^3 at 16:32 543.3 -> 530.8 us, 3072 x 4096 x
//    4096 545 -> 531, 4096 x 2048 x 4096 281.7 -> 275.7, V = 64 547 -> 533);
//    the 256 x 256 16-wave tile is still tried second.  At N = M (stages of
//    32 compressed rows) the 16-wave tiles take the place of the 8-wave
//    ones where they fill one round: 256 x 256 (4096^3 1029.7 -> 1025.5 us;
//    128 x 512 measured 1038), else 128 x 256 (2048 x 4096 x 4096 564.2 ->
//    554.7);
//  * else the 256 x 256 tile for dense-ish levels (N/M >= 1/2) and the
//    128 x 512 tile with 32 x 32 MFMAs for the sparser ones, unless its grid
//    would leave more than a quarter of the chip idle in the last wave, where
//    the 128 x 256 tile with 32 x 32 MFMAs (two workgroups per CU) is tried
//    first.
int preferences(int64_t m, int64_t n, int N, int M, int V, const TileInfo **out)
{
    int c = 0;
    auto add = [&](const char *name) { out[c++] = tile_by_name(name); };
    if (m <= 128) {
        add("16x512"); add("64x512"); add("128x128");
        return c;
    }
    if (m < 1024 || n < 1024) {
        add("128x256m32"); add("128x128"); add("128x512"); add("256x256");
        return c;
    }
    if ((2 * N <= M || N == M) && V % 32 == 0) {
        auto one_round = [&](const char *name) {
            const TileInfo &t = *tile_by_name(name);
            const int64_t tiles = ((m + t.BM - 1) / t.BM) * ((n + t.BN - 1) / t.BN);
            return tiles <= 256 && occupancy_of_grid(t, m, n) >= 0.75;
        };
        if (2 * N <= M && one_round("128x512m32w16")) add("128x512m32w16");
        else if (2 * N >= M && one_round("256x256m32w16")) add("256x256m32w16");
        else if (one_round("128x256m32w16")) add("128x256m32w16");
    }
    const char *big = 2 * N >= M ? "256x256" : "128x512m32";
    if (occupancy_of_grid(*tile_by_name(big), m, n) < 0.75) add("128x256m32");
    add(big);
    if (2 * N >= M) { add("128x512m32"); } else { add("256x256"); }
    add("128x512"); add("128x128");
    return c;
}

// The streaming kernel re-reads Bc once per 16 rows of C (mostly from L2 and
// the Infinity Cache), the tiled kernel once per 128 or more.  On MI355X the
// streaming kernel is faster up to 128 rows at k = n = 8192, and on products
// up to 1024 rows with m * w at most 2^20, where the tiled kernel's grid would
// be mostly split-k.  Measured (graph replay, per call) against the tiled
// kernel with split-k: 512 x 1024 x 1024 at N = M 40.7 -> 21.2 us, 512 x 2048
// x 2048 at N = M 66.6 -> 57.2 and at 16:32 50.3 -> 35.1, 1024 x 2048 x 2048
// at 16:32 69.3 -> 64.0, 12:32 63.0 -> 52.8, 8:32 52.3 -> 43.4; at N = M
// (m * w = 2^21) the tiled kernel stays ahead (101.0 against 103.2).
bool prefer_streaming(int64_t m, int64_t k, int N, int M)
{
    const int64_t w = (k / M) * N;
    return m <= 128 || (m <= 1024 && m * w <= (int64_t(1) << 20));
}

// Overrides of the dispatch rules, for tuning sweeps and the forced-variant
// tests only.  They come from the tuning string of the *_tuned entry points
// ("KEY=VALUE" pairs separated by commas); the default entry points use none
// and read no environment.  0 (or -1 for PS and GATHER, null for TILE) means
// "no override".
struct Tuning {
    char tile[24] = {};          // TILE: a tile name, or "skinny" for the streaming kernels
    int ka = 0;                  // KA: stage depth of the tiled kernel (32, 64, 128)
    int splits = 0;              // SPLITS: k split of any kernel
    int qpw = 0, skcols = 0, rt = 0;            // QPW, SKCOLS, RT: register-operand streaming kernel
    int ps = -1;                 // PS: 0 never the pipelined streaming kernel, 1 wherever it runs
    int psrt = 0, psbv = 0, pscpw = 0, psrb = 0;  // PSRT, PSBV, PSCPW, PSRB: its variant
    int gather = -1;             // GATHER: 0 never the direct-gather kernel, 1 wherever it runs
    int gct = 0, gnw = 0, gd = 0;  // GCT, GNW, GD: its variant
    int gh = 0;                  // GH: 1 one workgroup per strip, 2 row halves of 64 rows (above 64 rows)
    int rg = -1;                 // RG: 0 never the row-gather kernel, 1 wherever it runs
    int rgct = 0, rgnw = 0, rgd = 0;  // RGCT, RGNW, RGD: its variant
    const char *tile_or_null() const { return tile[0] ? tile : nullptr; }
};

const Tuning kNoTuning{};

// Parse a tuning string; false on an unknown key or a malformed pair.
bool parse_tuning(const char *spec, Tuning &t)
{
    t = Tuning{};
    if (!spec) return true;
    const char *s = spec;
    while (*s) {
        const char *eq = std::strchr(s, '=');
        if (!eq) return false;
        const char *end = std::strchr(eq + 1, ',');
        if (!end) end = eq + std::strlen(eq);
        const std::size_t klen = (std::size_t)(eq - s), vlen = (std::size_t)(end - eq - 1);
        char key[16] = {}, val[24] = {};
        if (klen == 0 || klen >= sizeof key || vlen == 0 || vlen >= sizeof val) return false;
        std::memcpy(key, s, klen);
        std::memcpy(val, eq + 1, vlen);
        if (std::strcmp(key, "TILE") == 0) {
            std::memcpy(t.tile, val, vlen + 1);
        } else {
            char *stop = nullptr;
            const long v = std::strtol(val, &stop, 10);
            if (*stop != '\0' || v < -1 || v > (1 << 20)) return false;
            struct { const char *name; int *field; } const fields[] = {
                {"KA", &t.ka}, {"SPLITS", &t.splits}, {"QPW", &t.qpw}, {"SKCOLS", &t.skcols},
                {"RT", &t.rt}, {"PS", &t.ps}, {"PSRT", &t.psrt}, {"PSBV", &t.psbv},
                {"PSCPW", &t.pscpw}, {"PSRB", &t.psrb}, {"GATHER", &t.gather}, {"GCT", &t.gct},
                {"GNW", &t.gnw}, {"GD", &t.gd}, {"RG", &t.rg}, {"RGCT", &t.rgct}, {"RGNW", &t.rgnw},
                {"RGD", &t.rgd}, {"GH", &t.gh}};
            bool found = false;
            for (const auto &f : fields)
                if (std::strcmp(key, f.name) == 0) { *f.field = (int)v; found = true; }
            if (!found) return false;
        }
        s = *end ? end + 1 : end;
    }
    return true;
}

// k short enough that the register-operand streaming kernel narrows its
// column tiles to fill the grid (at most two A chunks of 16 rows).
bool skinny_narrow_k(int64_t k) { return k <= 2 * skinny_chunk_cols(1); }

// Streaming kernel for short products: every Bc value is loaded once per
// 16 rows of C straight into MFMA operands and the A slice is staged in LDS;
// k is split across workgroups until the grid has about one workgroup per CU.
bool plan_skinny(const float *A, const float *Bc, const float *C, int64_t m, int64_t n, int64_t k,
                 int N, int M, int V, const Tuning &t, Plan &p)
{
    if (V % 16 != 0 || M % 4 != 0) return false;
    if (!aligned(A, 16) || !aligned(Bc, 16) || !aligned(C, 16)) return false;
    // 32 rows per workgroup (Bc read once per 32 rows instead of 16) when
    // that grid alone gives a workgroup per CU at 128 columns; measured on
    // MI355X: 1024 x 2048 x 2048 at 4:32 41 -> 32 us, 512 x 2048 x 2048 at
    // 8:32 30 -> 26 us.  Where the 32-row grid would need split-k it
    // measured slower.
    int rt = m >= 512 && ((m + 31) / 32) * ((n + 127) / 128) >= 256 ? 2 : 1;
    const int fr = t.rt;
    if (fr == 1 || fr == 2) rt = fr;
    if (M > skinny_chunk_cols(rt)) return false;
    // buffer offsets: the workgroup's rows of A and 4 rows of Bc per resource
    if ((int64_t)skinny_rows(rt) * k * 4 >= (int64_t(1) << 31)) return false;
    // Bc byte offsets inside a chunk (at most 1024 rows, plus a quad)
    if ((int64_t)1028 * n * 4 >= (int64_t(1) << 31)) return false;
    // 256 columns per workgroup when that already gives a workgroup per CU,
    // else 128 (and split-k for the rest)
    const int64_t tiles_m = (m + skinny_rows(rt) - 1) / skinny_rows(rt);
    int cols = tiles_m * ((n + 255) / 256) >= 256 ? 256 : 128;
    // A short k (each workgroup walks at most two A chunks): narrower
    // columns instead, down to 32, while the grid stays within one workgroup
    // per CU.  Each column tile re-reads the A slice from L2, which costs
    // little at this k, and the fuller grid hides the load latency.  Measured
    // on MI355X (graph replay): 256 x 256 x 256 at 16:32 8.4 -> 5.5 us (32
    // columns), 512 x 512 x 512 at 16:32 10.3 -> 8.0 and at N = M 12.6 ->
    // 10.2 (64), 256 x 512 x 1024 at 16:32 11.0 -> 8.6 (32), 128 x 2048 x 2048
    // at 4:32 10.9 -> 8.7 (64), 16 x 8192 x 1024 at 4:32 8.1 -> 6.0 (32).
    // Where k spans more chunks the split-k grid of 128 columns stays ahead
    // (16 rows, k = n = 4096 at 4:32: 9.4 against 11.7 us; k = n = 8192:
    // 14.3 against 19.0).
    if (rt == 1 && skinny_narrow_k(k))
        while (cols > 32 && tiles_m * ((n + cols / 2 - 1) / (cols / 2)) <= 256) cols /= 2;
    const int fc = t.skcols;
    if (fc == 32 || fc == 64 || fc == 128 || fc == 256) cols = fc;
    const int bv = std::min(bv_for(16, V), cols / 16);
    const int64_t tiles_n = (n + cols - 1) / cols;
    if (tiles_m * tiles_n > (1 << 24)) return false;
    const int64_t G = k / M, ntiles = tiles_m * tiles_n;
    // about one workgroup per CU, but at least 32 compressed rows (one quad
    // per wave) per workgroup; none when a workgroup's whole product is under
    // 2^21 flops, where the zero fill and the atomics cost more than the
    // fuller grid gives (graph replay: 512 x 512 x 512 at 16:32 10.8 ->
    // 10.3 us, at 8:32 9.7 -> 8.6, 256 x 256 x 256 at 16:32 8.9 -> 8.4; at
    // N = M, 2^21 flops per workgroup, split 2 stays ahead, 12.6 against 13.7)
    int64_t splits = std::min<int64_t>((256 + ntiles - 1) / ntiles, G * N / 32);
    splits = std::max<int64_t>(1, std::min<int64_t>(splits, 64));
    if (2 * skinny_rows(rt) * (int64_t)cols * (G * N) < (int64_t(1) << 21)) splits = 1;
    const int fs = t.splits;
    if (fs >= 1) splits = std::min<int64_t>(fs, std::max<int64_t>(G, 1));
    // longer runs per wave when each workgroup walks all of k
    int qpw = splits == 1 && skinny_has(rt, bv, 4, cols) ? 4 : skinny_has(rt, bv, 2, cols) ? 2 : 1;
    const int fq = t.qpw;
    if (skinny_has(rt, bv, fq, cols)) qpw = fq;
    if (!skinny_has(rt, bv, qpw, cols) || ntiles * splits > INT32_MAX) return false;
    p.kind = Kind::Skinny;
    p.BV = bv;
    p.QPW = qpw;
    p.COLS = cols;
    p.CW = skinny_chunk_cols(rt) / M;
    p.RT = rt;
    p.splits = (int)splits;
    p.tiles_m = (int)tiles_m;
    p.tiles_n = (int)tiles_n;
    return true;
}

// Pipelined streaming kernel: loader waves stream A, Bc and the offsets into
// an LDS ring several stages ahead of the compute waves.  Measured on MI355X
// against the register-operand streaming kernel: 64 x 8192 x 8192 at 4:32
// 29.1 -> 26.6 us, 128 x 8192 x 8192 42.5 -> 39.1, 1024 x 2048 x 2048 32.9 ->
// 20.4, 512 x 2048 x 2048 18.6 -> 15.3, 512 x 512 x 512 9.6 -> 7.0; at 8:32
// 512 x 2048 x 2048 24.3 -> 21.7.  It loses at 16 rows (the 16-row decode
// shapes keep the other kernel) and gains nothing at the denser levels.
// `force` (tuning sweeps and tests) takes it wherever it can run.
bool plan_stream(const float *A, const float *Bc, const float *C, int64_t m, int64_t n, int64_t k,
                 int N, int M, int V, bool force, const Tuning &t, Plan &p)
{
    const int KS = stream_stage_cols();
    if (V % 16 != 0 || M % 4 != 0 || M > KS) return false;
    if (!aligned(A, 16) || !aligned(Bc, 16) || !aligned(C, 16)) return false;
    // compressed rows per stage: the smallest ring row count that holds a
    // whole stage of KS/M windows, else the largest
    int rb = 64;
    for (int r : {16, 32, 64})
        if ((KS / M) * N <= r) { rb = r; break; }
    const int frb = t.psrb;
    if (frb == 16 || frb == 32 || frb == 64) rb = frb;
    if (N > rb) return false;
    if (!force && (rb > 32 || m <= 16)) return false;
    const int sw = std::min(KS / M, rb / N);
    const int64_t G = k / M;
    const int64_t nstages = (G + sw - 1) / sw;
    const int bvmax = std::min(bv_for(16, V), 2);
    auto ntiles = [&](int rt, int bv) {
        return ((m + stream_rows(rt) - 1) / stream_rows(rt)) * ((n + stream_cols(bv, 1) - 1) / stream_cols(bv, 1));
    };
    // Short products: 32-row tiles, k split until about one workgroup per
    // CU.  Taller ones: the largest tile whose grid alone fills the chip,
    // else the smallest, without split-k (their k is short: splitting it
    // measured slower).
    int rt = 2, bv = bvmax;
    bool fill_splits = m <= 128;
    if (m > 128) {
        const int order[][2] = {{2, 2}, {1, 2}, {1, 1}};
        rt = 1;
        bv = 1;
        for (const auto &o : order)
            if (o[1] <= bvmax && ntiles(o[0], o[1]) >= 256) {
                rt = o[0];
                bv = o[1];
                break;
            }
    }
    const int frt = t.psrt;
    if (frt == 1 || frt == 2 || frt == 4) rt = frt;
    const int fbv = t.psbv;
    if ((fbv == 1 || fbv == 2 || fbv == 4) && V % (16 * fbv) == 0) bv = fbv;
    int cpw = 1;
    const int fcp = t.pscpw;
    if (fcp == 1 || fcp == 2) cpw = fcp;
    if (!stream_has(rt, bv, cpw, rb)) return false;
    if ((int64_t)stream_rows(rt) * k * 4 >= (int64_t(1) << 31)) return false;
    if ((int64_t)rb * n * 4 >= (int64_t(1) << 31)) return false;
    const int cols = stream_cols(bv, cpw);
    const int64_t tiles_m = (m + stream_rows(rt) - 1) / stream_rows(rt);
    const int64_t tiles_n = (n + cols - 1) / cols;
    if (tiles_m * tiles_n > (1 << 24)) return false;
    const int64_t tiles = tiles_m * tiles_n;
    int64_t splits = 1;
    if (fill_splits)   // at least two stages per workgroup
        splits = std::max<int64_t>(1, std::min<int64_t>({(256 + tiles - 1) / tiles, nstages / 2, 64}));
    const int fs = t.splits;
    if (fs >= 1) splits = std::min<int64_t>(fs, std::max<int64_t>(G, 1));
    if (tiles * splits > INT32_MAX) return false;
    p.kind = Kind::Stream;
    p.RT = rt;
    p.BV = bv;
    p.CPW = cpw;
    p.RB = rb;
    p.SW = sw;
    p.COLS = cols;
    p.splits = (int)splits;
    p.tiles_m = (int)tiles_m;
    p.tiles_n = (int)tiles_n;
    return true;
}

// Row-gather kernel: up to 32 rows, one launch, every output written once.
// By default for at most 4 rows where its 32-column strips alone fill the
// chip: each quad then gathers at most 4 lines of A, and the single launch
// beats the streaming kernel's zero fill and split-k atomics.  Measured on
// MI355X (graph replay, against the register-operand streaming kernel with
// split-k): k = n = 8192 at 4:32, V = 64: 1 row 13.0 -> 10.9 us, 2 rows 13.1
// -> 11.3, 4 rows 13.2 -> 12.2; 4 x 11008 x 4096 at 8:32 27.4 -> 21.9.  From
// 8 rows on the gathered lines cost more than the launch and atomics they
// save (8 rows 13.4 against 13.9 us, 16 rows 14.2 against 18.0), and with
// fewer strips the grid does not fill the chip (1 x 4096 x 4096 at 8:32,
// V = 32: 9.9 against 10.2).  `force` (tuning sweeps and tests) takes it
// wherever it can run.
bool plan_rowgather(const float *A, const float *Bc, const float *C, int64_t m, int64_t n, int64_t k, int N,
                    int M, int V, bool force, const Tuning &t, Plan &p)
{
    if (m > 32 || k == 0 || !aligned(A, 4) || !aligned(Bc, 16) || !aligned(C, 4)) return false;
    if (!force && (m > 4 || n / 32 < 256)) return false;
    RowGatherCfg c{m <= 16 ? 1 : 2, 2, 8, 4};
    if (t.rgct) c.CT = t.rgct;
    if (t.rgnw) c.NW = t.rgnw;
    if (t.rgd) c.D = t.rgd;
    if (!rowgather_fits(c, m, n, k, N, M, V)) return false;
    p.kind = Kind::RowGather;
    p.RT = c.RT;
    p.CT = c.CT;
    p.NW = c.NW;
    p.D = c.D;
    p.splits = 1;
    p.tiles_m = 1;
    p.COLS = 16 * c.CT;
    p.tiles_n = (int)(n / p.COLS);
    return true;
}

Plan make_plan(const float *A, const float *Bc, const float *C, int64_t m, int64_t n, int64_t k,
               int N, int M, int V, const Tuning &t)
{
    Plan p;
    if (m == 0 || n == 0) return p;
    const char *force_tile = t.tile_or_null();
    const bool want_skinny =
        force_tile ? std::strcmp(force_tile, "skinny") == 0 : prefer_streaming(m, k, N, M);
    if (want_skinny) {
        if (t.rg != 0 && plan_rowgather(A, Bc, C, m, n, k, N, M, V, t.rg == 1, t, p)) return p;
        // the PS override (tuning sweeps and tests): 0 never takes the
        // pipelined streaming kernel, 1 takes it wherever it can run.  By
        // default it is not taken for up to 128 rows when k is short and
        // 128-column tiles would not fill the chip: the register-operand
        // kernel's narrowed tiles are faster there (128 x 2048 x 2048 at 4:32
        // 12.3 -> 8.7 us, 64 x 2048 x 2048 10.8 -> 7.8).
        const int ps = t.ps;
        const bool narrow_first = m <= 128 && skinny_narrow_k(k) && ((m + 15) / 16) * ((n + 127) / 128) < 256;
        if ((ps == 1 || (ps < 0 && !narrow_first)) && plan_stream(A, Bc, C, m, n, k, N, M, V, ps == 1, t, p))
            return p;
        if (plan_skinny(A, Bc, C, m, n, k, N, M, V, t, p)) return p;
    }
    p.kind = Kind::General;
    if (k % 4 != 0 || V % 16 != 0 || 128 % M != 0) return p;
    if (!aligned(A, 16) || !aligned(Bc, 16)) return p;
    // per-stage Bc buffer offsets reach (padded rows) x n x 4 bytes < 32 x n x 4
    if ((int64_t)32 * n * 4 >= (int64_t(1) << 31)) return p;

    // Stage depth: the smallest KA (a multiple of 32 and of M) whose stage
    // holds at least 16 compressed rows (8 for the tiles with few
    // accumulators per lane on grids of more tiles than CUs: they share a CU
    // between two workgroups and want a small LDS ring), so every stage
    // carries enough MFMA work to cover its fixed cost; deeper ones are tried
    // if it does not fit.
    auto ka_list = [&](int min_rows, int *order) {
        int cnt = 0;
        for (int KA : {32, 64, 128})
            if (KA % M == 0 && (KA / M) * N >= min_rows) order[cnt++] = KA;
        for (int KA : {128, 64, 32})
            if (KA % M == 0 && (KA / M) * N < min_rows) order[cnt++] = KA;
        return cnt;
    };
    // The 16-wave tiles take stages of exactly 32 compressed rows where
    // those fit (their 16-row A chunks leave the registers for them): half as
    // many barriers per MFMA.  Measured (per-launch events): 2048 x 4096 x 4096 at
    // 16:32 on 128 x 256 tiles 300.2 -> 292.0 us (KA = 64).
    int ka_order[3], ka_small[3], ka_deep[4];
    int nka = ka_list(16, ka_order), nks = ka_list(8, ka_small), nkd = 0;
    for (int KA : {32, 64, 128})   // a whole stage of 32 rows, no padding, then the usual order
        if (KA % M == 0 && (KA / M) * N == 32) ka_deep[nkd++] = KA;
    for (int i = 0; i < nka; ++i) ka_deep[nkd++] = ka_order[i];
    const int ka_force = t.ka;
    if (ka_force == 32 || ka_force == 64 || ka_force == 128) {
        ka_order[0] = ka_small[0] = ka_deep[0] = ka_force;
        nka = nks = nkd = 1;
    }

    const TileInfo *cand[8];
    int nc = preferences(m, n, N, M, V, cand);
    if (force_tile) {
        const TileInfo *t = tile_by_name(force_tile);
        if (t) { cand[0] = t; nc = 1; }
    }
    // first tile shape (in preference order) that some stage depth fits
    const TileInfo *tile = nullptr;
    int KA = 0, NQ = 0, BV = 0;
    for (int j = 0; j < nc && !tile; ++j) {
        if (!cand[j]) continue;
      // the widest column group first; narrower ones where a wave's tile is
      // narrower than MI * bv
      for (int bv = bv_for(cand[j]->MI, V); bv >= 1 && !tile; bv /= 2) {
        if (!aligned(C, 4 * bv)) continue;
        // the shallow rule pays off only when the grid has more tiles than
        // CUs, so that a second workgroup per CU has work to bring
        const int64_t tiles_c = ((m + cand[j]->BM - 1) / cand[j]->BM) * ((n + cand[j]->BN - 1) / cand[j]->BN);
        const bool small = two_per_cu(*cand[j]) && tiles_c > 256;
        const bool deep = cand[j]->waves == 16;
        const int *order = small ? ka_small : deep ? ka_deep : ka_order;
        const int norder = small ? nks : deep ? nkd : nka;
        for (int i = 0; i < norder && !tile; ++i) {
            const int nq = stage_nq(order[i], (order[i] / M) * N);
            if (nq != 0 && tile_ok(*cand[j], bv, order[i], nq, k, V)) {
                tile = cand[j];
                KA = order[i];
                NQ = nq;
                BV = bv;
            }
        }
      }
    }
    if (!tile) return p;

    const int64_t tiles_m = (m + tile->BM - 1) / tile->BM, tiles_n = (n + tile->BN - 1) / tile->BN;
    const int64_t groups = k / M, gps = KA / M;
    const int64_t stages = (groups + gps - 1) / gps;
    if (tiles_m * tiles_n > (1 << 24) || stages > INT32_MAX) return p;
    const int64_t ntiles = tiles_m * tiles_n;
    // split k until the grid has about one workgroup per CU (half that for
    // the thinnest products, where fewer, longer k slices stream better)
    const int64_t target = m <= 16 ? 128 : 256;
    int64_t splits = 1;
    if (ntiles < target && stages > 1) {
        splits = std::min<int64_t>({(target + ntiles - 1) / ntiles, stages, 32});
        // The 16-wave tiles run one workgroup per CU: a split that overflows
        // one round leaves a partial second one, so they split only into
        // whole rounds.  Measured on MI355X at 8:32, k = 4096 (graph replay):
        // 1536 x 4096 on 192 tiles of 128 x 256 199.6 -> 165.0 us without
        // the split, 2048 x 2816 on 176 tiles 196.5 -> 165.1.
        if (tile->waves == 16) splits = std::max<int64_t>(1, std::min<int64_t>(splits, target / ntiles));
    }
    if (t.splits >= 1) splits = std::min<int64_t>(t.splits, std::max<int64_t>(stages, 1));

    // Two column regions where the sparse levels' wide 16-wave tile would
    // need more than one round but the rest fits in one: whole 128 x 512
    // column tiles for one round, then the remaining columns as one round of
    // the 128 x 256 16-wave tile, a second launch, neither split.  Measured
    // on MI355X (2048 x 11008 x 4096 at 8:32, per-launch events): the two
    // regions alone take 284.9 us (2048 x 8192) and 165.1 us (2048 x 2816),
    // against 474.8 us for the 128 x 256 8-wave tile over the whole grid
    // (688 tiles, two per CU); at 4:32 260.3 against 362.8.  At 12:32 and
    // 16:32 the 8-wave tile stays ahead (670 against 686 us, 832 against 858
    // for the two regions timed alone).
    if (!force_tile && !ka_force && t.splits < 1 && 4 * N <= M && V % 32 == 0 && m >= 1024 && n >= 1024) {
        const TileInfo *big = tile_by_name("128x512m32w16"), *rest = tile_by_name("128x256m32w16");
        const int64_t tm = (m + big->BM - 1) / big->BM;
        const int64_t big_tiles = tm * ((n + big->BN - 1) / big->BN);
        const int64_t cols1 = std::min<int64_t>(256 / tm, n / big->BN) * big->BN;
        const int64_t tn2 = (n - cols1 + rest->BN - 1) / rest->BN;
        auto fit = [&](const TileInfo *tl, int &bv_out, int &ka_out, int &nq_out) {
            for (int bv = bv_for(tl->MI, V); bv >= 1; bv /= 2) {
                if (!aligned(C, 4 * bv)) continue;
                for (int i = 0; i < nka; ++i) {
                    const int nq = stage_nq(ka_order[i], (ka_order[i] / M) * N);
                    if (nq != 0 && tile_ok(*tl, bv, ka_order[i], nq, k, V)) {
                        bv_out = bv;
                        ka_out = ka_order[i];
                        nq_out = nq;
                        return true;
                    }
                }
            }
            return false;
        };
        int bv1 = 0, ka1 = 0, nq1 = 0, bv2 = 0, ka2 = 0, nq2 = 0;
        // the second round must keep most of the chip busy (R4's keeps 176
        // CUs): a nearly empty one costs a whole round's time
        if (big_tiles > 256 && big_tiles <= 512 && cols1 > 0 && cols1 < n && cols1 % V == 0 && tm * tn2 <= 256 &&
            tm * tn2 >= 160 &&
            fit(big, bv1, ka1, nq1) && fit(rest, bv2, ka2, nq2)) {
            p.kind = Kind::Tiled;
            p.tile = big;
            p.BV = bv1;
            p.KA = ka1;
            p.NQ = nq1;
            p.RS = (ka1 / M) * N;
            p.stages = (int)((groups + ka1 / M - 1) / (ka1 / M));
            p.splits = 1;
            p.tiles_m = (int)tm;
            p.tiles_n = (int)(cols1 / big->BN);
            p.tile2 = rest;
            p.BV2 = bv2;
            p.KA2 = ka2;
            p.NQ2 = nq2;
            p.stages2 = (int)((groups + ka2 / M - 1) / (ka2 / M));
            p.tiles_n2 = (int)tn2;
            p.col_split = cols1;
            return p;
        }
    }
    p.kind = Kind::Tiled;
    p.tile = tile;
    p.BV = BV;
    p.KA = KA;
    p.NQ = NQ;
    p.RS = (KA / M) * N;
    p.stages = (int)stages;
    p.splits = (int)splits;
    p.tiles_m = (int)tiles_m;
    p.tiles_n = (int)tiles_n;
    return p;
}

// Direct-gather kernel (workspace entry point only): short products whose
// column blocks hold whole strips.  k is split across workgroups until the
// grid has about one workgroup per CU, keeping at least 8 quads per wave.
// Measured on MI355X at k = n = 8192, 4:32, V = 64 (graph replay, against
// the streaming kernels through the same workspace): 64 rows 26.3 -> 22.1 us,
// 128 rows 41.0 -> 33.1; at 16 rows it lost (16.4 against 15.0), and split-k
// through its partial strips lost everywhere it was tried.
bool plan_gather(const float *Bc, int64_t m, int64_t n, int64_t k, int N, int M, int V, bool force,
                 const Tuning &t, Plan &p)
{
    if (k == 0 || m > 128 || !aligned(Bc, 16)) return false;
    if (!force && (m <= 16 || !prefer_streaming(m, k, N, M))) return false;
    GatherCfg c;
    c.RT = m <= 16 ? 1 : m <= 32 ? 2 : m <= 64 ? 4 : 8;
    // {CT, NW, D} per RT.  A shallow ring measured faster than a deep one
    // (64 x 8192 x 8192 at 4:32: D = 8 21.7 us, D = 4 20.1-21.5, D = 2 21.9;
    // 128 rows: D = 8 33.0, D = 4 32.2): more loads in flight mostly queue.
    static const int defaults[9][3] = {{}, {2, 8, 4}, {2, 8, 4}, {}, {2, 8, 4}, {}, {}, {}, {2, 4, 4}};
    c.CT = t.gct ? t.gct : defaults[c.RT][0];
    c.NW = t.gnw ? t.gnw : defaults[c.RT][1];
    c.D = t.gd ? t.gd : defaults[c.RT][2];
    if (!gather_has(c) || V % (16 * c.CT) != 0) return false;
    const int64_t w = (k / M) * N, strips = n / (16 * c.CT);
    const int64_t nquads = (w + 3) / 4;
    // At offsets, and Bc offsets up to the quads the register ring loads
    // ahead of the last one (D <= 16)
    if (k * gather_rows(c.RT) * 4 >= (int64_t(1) << 31)) return false;
    if ((4 * nquads + 4 * 2 * 16 + 4) * n * 4 >= (int64_t(1) << 31)) return false;
    if ((n / V) * w >= (int64_t(1) << 29) || strips > (1 << 24)) return false;
    // By default only where the strips alone fill the chip: its fixed costs
    // (the transposition pass, two dependent loads before the first MFMA)
    // pay off on long strips, and its split-k through partial strips loses
    // to the streaming kernels.  Measured (graph replay, against the best
    // streaming variant): 64 x 8192 x 8192 at 8:32 29.7 against 35.5 us,
    // 128 x 8192 x 2048 at 4:32 15.7 against 18.9, 64 x 11008 x 4096 at 8:32
    // 28.9 against 46.9; with split-k 128 x 4096 x 4096 at 4:32 20.8 against
    // 17.1, 32 x 4096 x 4096 at 8:32 14.4 against 12.9, and on small products
    // 128 x 512 x 512 at 16:32 14.1 against 6.5.
    if (!force && strips < 256) return false;
    int64_t splits = 1;
    if (strips < 256)
        splits = std::max<int64_t>(1, std::min<int64_t>((256 + strips - 1) / strips, nquads / (8 * c.NW)));
    const int fs = t.splits;
    if (fs >= 1) splits = std::min<int64_t>(fs, std::max<int64_t>(nquads, 1));
    // Above 64 rows without split-k, on short strips: two row halves of 64
    // rows, each a workgroup of the 64-row variant (two per CU; the halves of
    // a strip share its Bc lines through one XCD's L2), where the 128-row
    // variant has one wave per SIMD and few trips of its ring.  Measured
    // (graph replay, m x k x n): at w <= 512 compressed rows on 256 strips
    // 128 x 1024 x 8192 at 4:32 12.8 -> 11.2 us, 128 x 2048 x 8192 15.5 ->
    // 13.8, 80 x 2048 x 8192 14.7 -> 13.4, 72 x 3072 x 8192 17.3 -> 16.0,
    // 128 x 4096 x 8192 20.7 -> 19.3, 128 x 2048 x 8192 at 8:32 19.9 -> 18.2;
    // slower at w = 1024 (128 x 8192 x 8192 at 4:32 29.5 -> 30.8) and where
    // the doubled grid no longer fits two workgroups per CU (128 x 4096 x
    // 16384 at 4:32 29.6 -> 31.7).
    // (A forced variant, GCT / GNW / GD, keeps one workgroup per strip unless
    // GH = 2 asks for the halves.)
    const bool halves = t.gh == 2 || (t.gh == 0 && !t.gct && !t.gnw && !t.gd && w <= 512 && strips <= 256);
    if (halves && m > 64 && splits == 1) {
        GatherCfg h = c;
        h.RT = 4;
        h.H = 2;
        h.CT = t.gct ? t.gct : defaults[4][0];
        h.NW = t.gnw ? t.gnw : defaults[4][1];
        h.D = t.gd ? t.gd : defaults[4][2];
        if (gather_has(h) && V % (16 * h.CT) == 0 && n / (16 * h.CT) == strips) c = h;
    }
    if (strips * splits * c.H > INT32_MAX) return false;
    p.kind = Kind::Gather;
    p.RT = c.RT;
    p.CT = c.CT;
    p.NW = c.NW;
    p.D = c.D;
    p.H = c.H;
    p.splits = (int)splits;
    p.tiles_m = 1;
    p.tiles_n = (int)strips;
    p.COLS = 16 * c.CT;
    p.ws_bytes = gather_layout(c, n, k, N, M, V, (int)splits).total;
    return true;
}

// The plan of a call that brings a workspace.  The GATHER override (tuning
// sweeps and tests): 0 never takes the direct-gather kernel, 1 takes it
// wherever it can run.
Plan make_ws_plan(const float *A, const float *Bc, const float *C, int64_t m, int64_t n, int64_t k, int N,
                  int M, int V, const Tuning &t)
{
    Plan p;
    if (m == 0 || n == 0) return p;
    const int g = t.gather;
    if (g != 0 && plan_gather(Bc, m, n, k, N, M, V, g == 1, t, p)) return p;
    return make_plan(A, Bc, C, m, n, k, N, M, V, t);
}

hipError_t launch_general(const float *A, const float *Bc, const uint8_t *idx, float *C,
                          int64_t m, int64_t n, int64_t k, int N, int M, int V, const Epilogue &epi,
                          hipStream_t stream)
{
    const int64_t gx = (n + GEN_COLS - 1) / GEN_COLS;
    const int64_t gy = std::min<int64_t>((m + GEN_ROWS - 1) / GEN_ROWS, 65535);
    if (gx > INT32_MAX) return hipErrorInvalidValue;
    hipLaunchKernelGGL(nm_general_kernel, dim3((unsigned)gx, (unsigned)gy), dim3(GEN_COLS), 0,
                       stream, A, Bc, idx, C, m, n, k, N, M, V, epi);
    return hipGetLastError();
}

bool trivial(const Epilogue &e) { return e.alpha == 1.f && !e.bias && e.act == NMSPMM_ACT_NONE; }

// `ws` (plan_ws_bytes(p) bytes) or null: split-k through atomic adds into a
// zeroed C.
hipError_t launch_main(const Plan &p, const float *A, const float *Bc, const uint8_t *idx, float *C,
                       int64_t m, int64_t n, int64_t k, int N, int M, int V, const Epilogue &epi,
                       void *ws, hipStream_t stream)
{
    if (p.kind == Kind::General)
        return launch_general(A, Bc, idx, C, m, n, k, N, M, V, epi, stream);
    float *ws_part = static_cast<float *>(ws);
    if (p.kind == Kind::Gather && !ws) return hipErrorInvalidValue;
    if (p.splits > 1 && !ws) {
        const int64_t count = m * n;
        if (aligned(C, 16)) {
            const int64_t blocks = std::min<int64_t>((count / 4 + 255) / 256 + 1, 4096);
            hipLaunchKernelGGL(nm_zero4_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, C, count);
        } else {
            const int64_t blocks = std::min<int64_t>((count + 255) / 256, 4096);
            hipLaunchKernelGGL(nm_zero_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, C, count);
        }
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (p.kind == Kind::Skinny) {
        SkinnyArgs s;
        s.A = A;
        s.Bc = Bc;
        s.idx = idx;
        s.C = C;
        s.m = m;
        s.n = n;
        s.k = k;
        s.N = N;
        s.M = M;
        s.V = V;
        s.splits = p.splits;
        s.tiles_m = p.tiles_m;
        s.tiles_n = p.tiles_n;
        s.cw = p.CW;
        s.epi = epi;
        // Bc streamed past L2: at least 16 MB, four XCDs' worth
        s.stream_b = (k / M) * N * n * 4 >= (int64_t(16) << 20) ? 1 : 0;
        return launch_skinny(p.RT, p.BV, p.QPW, p.COLS, s, stream);
    }
    if (p.kind == Kind::Gather) {
        GatherArgs g;
        g.A = A;
        g.Bc = Bc;
        g.idx = idx;
        g.C = C;
        g.m = m;
        g.n = n;
        g.k = k;
        g.N = N;
        g.M = M;
        g.V = V;
        g.splits = p.splits;
        g.epi = epi;
        g.ws = ws;
        g.halves = p.H;
        GatherCfg gc{p.RT, p.CT, p.NW, p.D};
        gc.H = p.H;
        return launch_gather(gc, g, stream);
    }
    if (p.kind == Kind::RowGather) {
        RowGatherArgs g;
        g.A = A;
        g.Bc = Bc;
        g.idx = idx;
        g.C = C;
        g.m = m;
        g.n = n;
        g.k = k;
        g.N = N;
        g.M = M;
        g.V = V;
        g.epi = epi;
        // Bc streamed past L2: at least 16 MB, four XCDs' worth
        g.stream_b = (k / M) * N * n * 4 >= (int64_t(16) << 20) ? 1 : 0;
        return launch_rowgather(RowGatherCfg{p.RT, p.CT, p.NW, p.D}, g, stream);
    }
    if (p.kind == Kind::Stream) {
        StreamArgs s;
        s.A = A;
        s.Bc = Bc;
        s.idx = idx;
        s.C = C;
        s.m = m;
        s.n = n;
        s.k = k;
        s.N = N;
        s.M = M;
        s.V = V;
        s.splits = p.splits;
        s.tiles_m = p.tiles_m;
        s.tiles_n = p.tiles_n;
        s.sw = p.SW;
        s.epi = epi;
        s.ws = ws_part;
        return launch_stream(p.RT, p.BV, p.CPW, p.RB, s, stream);
    }
    TiledArgs a;
    a.A = A;
    a.Bc = Bc;
    a.idx = idx;
    a.C = C;
    a.m = m;
    a.n = n;
    a.k = k;
    a.N = N;
    a.M = M;
    a.V = V;
    a.RS = p.RS;
    a.stages = p.stages;
    a.splits = p.splits;
    a.tiles_m = p.tiles_m;
    a.tiles_n = p.tiles_n;
    a.epi = epi;
    hipError_t e = p.tile->launch(p.BV, p.KA, p.NQ, a, stream);
    if (e != hipSuccess || !p.tile2) return e;
    // the second column region, with its own tile and stage depth
    a.RS = (p.KA2 / M) * N;
    a.stages = p.stages2;
    a.tiles_n = p.tiles_n2;
    a.col_begin = p.col_split;
    return p.tile2->launch(p.BV2, p.KA2, p.NQ2, a, stream);
}

// The kernel(s) of a plan, then, when k was split across workgroups and the
// epilogue does something, one pass over C that applies it.
hipError_t launch_plan(const Plan &p, const float *A, const float *Bc, const uint8_t *idx, float *C,
                       int64_t m, int64_t n, int64_t k, int N, int M, int V, const Epilogue &epi,
                       void *ws, hipStream_t stream)
{
    hipError_t e = launch_main(p, A, Bc, idx, C, m, n, k, N, M, V, epi, ws, stream);
    if (e == hipSuccess && ws && p.splits > 1) {
        const float *part = static_cast<const float *>(ws);
        int rows = stream_rows(p.RT);
        if (p.kind == Kind::Gather) {
            part += gather_layout(GatherCfg{p.RT, p.CT, p.NW, p.D}, n, k, N, M, V, p.splits).part / 4;
            rows = gather_rows(p.RT);
        }
        const int64_t blocks = std::min<int64_t>((m * n + 255) / 256, 8192);
        hipLaunchKernelGGL(nm_splitk_reduce_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, part, C, m,
                           n, rows, p.COLS, p.tiles_n, p.splits, epi);
        return hipGetLastError();
    }
    if (e == hipSuccess && p.kind == Kind::Gather) return e;
    if (e != hipSuccess || p.kind == Kind::General || p.splits == 1 || trivial(epi)) return e;
    const int64_t count = m * n;
    const int64_t blocks = std::min<int64_t>((count + 255) / 256, 4096);
    hipLaunchKernelGGL(nm_epilogue_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, C, count, n,
                       epi);
    return hipGetLastError();
}

}  // namespace
}  // namespace nmspmm

using namespace nmspmm;

namespace {

const char *plan_name(const Plan &p, bool with_ws)
{
    switch (p.kind) {
    case Kind::None: return "none";
    case Kind::General: return "nm_general_kernel";
    case Kind::Tiled: case Kind::Skinny: case Kind::Stream: case Kind::Gather: case Kind::RowGather: break;
    }
    thread_local char buf[160];
    if (p.kind == Kind::RowGather) {
        std::snprintf(buf, sizeof buf, "nm_rowgather_kernel<r%d,c%d,w%d,d%d>,split1", 16 * p.RT, p.COLS, p.NW, p.D);
        return buf;
    }
    if (p.kind == Kind::Gather && p.H > 1) {
        std::snprintf(buf, sizeof buf, "nm_gather_kernel<r%dx%d,c%d,w%d,d%d>+prep,split%d", gather_rows(p.RT), p.H,
                      p.COLS, p.NW, p.D, p.splits);
        return buf;
    }
    if (p.kind == Kind::Gather) {
        std::snprintf(buf, sizeof buf, "nm_gather_kernel<r%d,c%d,w%d,d%d>+prep,split%d", gather_rows(p.RT),
                      p.COLS, p.NW, p.D, p.splits);
        return buf;
    }
    if (p.kind == Kind::Stream && with_ws && p.splits > 1) {
        std::snprintf(buf, sizeof buf, "nm_stream_kernel<r%d,c%d,bv%d,rb%d>+ws,split%d", 16 * p.RT, p.COLS,
                      p.BV, p.RB, p.splits);
        return buf;
    }
    if (p.kind == Kind::Stream) {
        std::snprintf(buf, sizeof buf, "nm_stream_kernel<r%d,c%d,bv%d,rb%d>%s%d", 16 * p.RT, p.COLS,
                      p.BV, p.RB, p.splits > 1 ? "+zero,split" : ",split", p.splits);
        return buf;
    }
    if (p.kind == Kind::Skinny) {
        if (p.RT == 1)
            std::snprintf(buf, sizeof buf, "nm_skinny_kernel<c%d,bv%d,qpw%d>%s%d", p.COLS, p.BV, p.QPW,
                          p.splits > 1 ? "+zero,split" : ",split", p.splits);
        else
            std::snprintf(buf, sizeof buf, "nm_skinny_kernel<c%d,bv%d,qpw%d,rows%d>%s%d", p.COLS, p.BV,
                          p.QPW, 16 * p.RT, p.splits > 1 ? "+zero,split" : ",split", p.splits);
        return buf;
    }
    if (p.tile2) {
        std::snprintf(buf, sizeof buf,
                      "nm_tiled_kernel<%s,bv%d,ka%d,nq%d>,split1+cols%lld:nm_tiled_kernel<%s,bv%d,ka%d,nq%d>,split1",
                      p.tile->name, p.BV, p.KA, p.NQ, (long long)p.col_split, p.tile2->name, p.BV2, p.KA2, p.NQ2);
        return buf;
    }
    std::snprintf(buf, sizeof buf, "nm_tiled_kernel<%s,bv%d,ka%d,nq%d>%s%d", p.tile->name, p.BV,
                  p.KA, p.NQ, p.splits > 1 ? "+zero,split" : ",split", p.splits);
    return buf;
}

}  // namespace

extern "C" const char *nmspmm_kernel_name_tuned(int64_t m, int64_t n, int64_t k, int N, int M, int V,
                                                int with_workspace, const char *tuning)
{
    Tuning t;
    if (!parse_tuning(tuning, t) || !shape_ok(m, n, k, N, M, V) || !sizes_fit(m, n, k)) return "invalid";
    // assume buffers as aligned as the allocator returns them
    alignas(64) static const float probe[16] = {};
    if (with_workspace) return plan_name(make_ws_plan(probe, probe, probe, m, n, k, N, M, V, t), true);
    return plan_name(make_plan(probe, probe, probe, m, n, k, N, M, V, t), false);
}

extern "C" const char *nmspmm_kernel_name(int64_t m, int64_t n, int64_t k, int N, int M, int V)
{
    // outside graph capture nmspmm_run takes the workspace plan, with the stream's cached
    // workspace, where that plan is the direct-gather kernel
    const char *with_ws = nmspmm_kernel_name_tuned(m, n, k, N, M, V, 1, nullptr);
    if (std::strncmp(with_ws, "nm_gather_kernel<", 17) == 0) return with_ws;
    return nmspmm_kernel_name_tuned(m, n, k, N, M, V, 0, nullptr);
}

extern "C" const char *nmspmm_kernel_name_ws(int64_t m, int64_t n, int64_t k, int N, int M, int V)
{
    return nmspmm_kernel_name_tuned(m, n, k, N, M, V, 1, nullptr);
}

namespace nmspmm {
namespace {

// Argument checks of every product entry point (NMSPMM_OK: go on; m == 0 or
// n == 0 then means nothing to launch).
nmspmm_status_t check_run_args(const float *A, const float *Bc, const uint8_t *idx, const float *C, int64_t m,
                               int64_t n, int64_t k, int N, int M, int V, const float *bias, nmspmm_act_t act)
{
    if (!shape_ok(m, n, k, N, M, V)) return NMSPMM_ERR_INVALID_ARG;
    if (act != NMSPMM_ACT_NONE && act != NMSPMM_ACT_RELU && act != NMSPMM_ACT_GELU)
        return NMSPMM_ERR_INVALID_ARG;
    if (!sizes_fit(m, n, k)) return NMSPMM_ERR_UNSUPPORTED;
    if (m == 0 || n == 0) return NMSPMM_OK;
    if (!C) return NMSPMM_ERR_INVALID_ARG;
    if (k > 0 && (!A || !Bc || !idx)) return NMSPMM_ERR_INVALID_ARG;
    if (!aligned(C, 4) || (k > 0 && (!aligned(A, 4) || !aligned(Bc, 4))) || !aligned(bias, 4))
        return NMSPMM_ERR_UNSUPPORTED;
    return NMSPMM_OK;
}

// Workspaces of the calls that bring none (nmspmm_run, nmspmm_run_ex): one
// buffer per (device, stream), allocated on the first call that needs it
// (and again, larger, when a call needs more) and kept for the next calls on
// that stream.  Each call makes its stream wait for the event the buffer's
// previous user recorded after its kernels, and records it again after its
// own.  Calls on one stream are ordered anyway; the wait orders the first
// call on a stream whose handle reuses that of a destroyed one (HIP hands a
// new stream the last destroyed stream's handle) after the destroyed
// stream's last kernels.  The pair costs about 1.4 us of host time per call
// and no measurable GPU time (MI355X), where a stream-ordered allocation
// from a memory pool and its release cost 8.7 us and made back-to-back calls
// host-bound.  At
// most kWsEntries buffers are kept: a call past that releases the oldest
// idle entry's buffer once that entry's last kernels are done (an entry a
// call is between acquiring and marking is never released or regrown; a call
// that finds none it may use runs without a workspace).
constexpr int kWsEntries = 16;
struct WsEntry {
    int dev = -1;
    hipStream_t stream = nullptr;
    void *buf = nullptr;
    size_t bytes = 0;
    hipEvent_t done = nullptr;
    uint64_t used = 0;   // call counter of the last use (for the oldest entry)
    int busy = 0;        // calls between ws_acquire and ws_done (never dropped then)
};
WsEntry g_ws[kWsEntries];
uint64_t g_ws_calls = 0;
std::mutex g_ws_mu;

// Release an entry's buffer and event after its last kernels.
void ws_drop(WsEntry &e)
{
    if (e.done) (void)hipEventSynchronize(e.done);
    if (e.buf) (void)hipFree(e.buf);
    if (e.done) (void)hipEventDestroy(e.done);
    e = WsEntry{};
}

// A workspace of at least `need` bytes for a call on `stream` (the current
// device), ordered after the buffer's previous use; null when none can be
// had.  ws_done(...) must follow the call's launches.
void *ws_acquire(hipStream_t stream, size_t need, int *slot)
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) {
        (void)hipGetLastError();
        return nullptr;
    }
    std::lock_guard<std::mutex> lock(g_ws_mu);
    int hit = -1, oldest = -1;
    for (int i = 0; i < kWsEntries; ++i) {
        if (g_ws[i].buf && g_ws[i].dev == dev && g_ws[i].stream == stream) hit = i;
        if (g_ws[i].buf && g_ws[i].busy == 0 && (oldest < 0 || g_ws[i].used < g_ws[oldest].used)) oldest = i;
    }
    int i = hit;
    if (i >= 0 && g_ws[i].bytes < need) {
        if (g_ws[i].busy > 0) return nullptr;
        ws_drop(g_ws[i]);   // grow: the old buffer after its last use
    }
    if (i < 0) {
        for (int j = 0; j < kWsEntries && i < 0; ++j)
            if (!g_ws[j].buf) i = j;
        if (i < 0) {
            if (oldest < 0) return nullptr;
            i = oldest;
            ws_drop(g_ws[i]);
        }
    }
    WsEntry &e = g_ws[i];
    if (!e.buf) {
        const size_t bytes = (need + 255) / 256 * 256;
        if (hipMalloc(&e.buf, bytes) != hipSuccess) {
            e = WsEntry{};
            (void)hipGetLastError();
            return nullptr;
        }
        // completion order only: the next user overwrites the buffer before
        // reading it, so no system-scope fence (cache write-back) is needed
        if (hipEventCreateWithFlags(&e.done, hipEventDisableTiming | hipEventDisableSystemFence) != hipSuccess) {
            (void)hipFree(e.buf);
            e = WsEntry{};
            (void)hipGetLastError();
            return nullptr;
        }
        e.dev = dev;
        e.stream = stream;
        e.bytes = bytes;
    } else if (hipStreamWaitEvent(stream, e.done, 0) != hipSuccess) {
        (void)hipGetLastError();
        return nullptr;
    }
    e.used = ++g_ws_calls;
    ++e.busy;
    *slot = i;
    return e.buf;
}

// After the call's launches on `stream`: mark the buffer's last use.
hipError_t ws_done(int slot, hipStream_t stream)
{
    std::lock_guard<std::mutex> lock(g_ws_mu);
    --g_ws[slot].busy;
    return hipEventRecord(g_ws[slot].done, stream);
}

// Whether work on `stream` is being captured into a graph (or that cannot be
// told): such calls take no cached workspace.
bool capturing(hipStream_t stream)
{
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(stream, &cs) != hipSuccess) {
        (void)hipGetLastError();
        return true;
    }
    return cs != hipStreamCaptureStatusNone;
}

// `pooled`: a call whose workspace (if any) is smaller than its workspace
// plan needs takes the stream's cached workspace instead, outside graph
// capture, where that plan is the direct-gather kernel; when none can be
// had, the call runs the plan that takes none.  (Measured on MI355X, 2000
// back-to-back calls from C++ at 64 x 8192 x 8192, 4:32: caller workspace
// 15.5 us per call, the cached workspace 18.2, no workspace (split-k,
// atomics) 25.4; at 128 rows 26.4, 28.8 and 37.5.  The streaming kernels'
// split-k through a workspace gains less than the workspace costs and keeps
// its atomics there.)
nmspmm_status_t run_impl(const float *A, const float *Bc, const uint8_t *idx, float *C, int64_t m, int64_t n,
                         int64_t k, int N, int M, int V, float alpha, const float *bias, nmspmm_act_t act,
                         void *workspace, size_t ws_bytes, const Tuning &t, hipStream_t stream,
                         bool pooled = false)
{
    const nmspmm_status_t st = check_run_args(A, Bc, idx, C, m, n, k, N, M, V, bias, act);
    if (st != NMSPMM_OK || m == 0 || n == 0) return st;
    if (workspace && !aligned(workspace, 256)) return NMSPMM_ERR_UNSUPPORTED;
    int cached = -1;
    if (pooled) {
        const Plan pw = make_ws_plan(A, Bc, C, m, n, k, N, M, V, t);
        const int64_t need = pw.kind == Kind::Gather ? plan_ws_bytes(pw) : 0;
        if (need > 0 && (!workspace || (uint64_t)need > (uint64_t)ws_bytes) && !capturing(stream)) {
            void *buf = ws_acquire(stream, (size_t)need, &cached);
            if (buf) {
                workspace = buf;
                ws_bytes = (size_t)need;
            } else {
                cached = -1;
            }
        }
    }
    // with a workspace large enough for it, the plan of nmspmm_workspace_bytes;
    // otherwise that of a call without one
    Plan p = workspace ? make_ws_plan(A, Bc, C, m, n, k, N, M, V, t) : make_plan(A, Bc, C, m, n, k, N, M, V, t);
    if (workspace && (uint64_t)plan_ws_bytes(p) > (uint64_t)ws_bytes) p = make_plan(A, Bc, C, m, n, k, N, M, V, t);
    if (p.kind == Kind::None) {
        if (cached >= 0) (void)ws_done(cached, stream);
        return NMSPMM_OK;
    }
    Epilogue epi;
    epi.alpha = alpha;
    epi.bias = bias;
    epi.act = act;
    const int64_t need = plan_ws_bytes(p);
    void *ws = need > 0 && workspace && (uint64_t)need <= (uint64_t)ws_bytes ? workspace : nullptr;
    const hipError_t e = launch_plan(p, A, Bc, idx, C, m, n, k, N, M, V, epi, ws, stream);
    const hipError_t f = cached >= 0 ? ws_done(cached, stream) : hipSuccess;
    return e == hipSuccess && f == hipSuccess ? NMSPMM_OK : NMSPMM_ERR_HIP;
}

}  // namespace
}  // namespace nmspmm

extern "C" nmspmm_status_t nmspmm_run_ex(const float *A, const float *Bc, const uint8_t *idx,
                                         float *C, int64_t m, int64_t n, int64_t k, int N, int M,
                                         int V, float alpha, const float *bias, nmspmm_act_t act,
                                         hipStream_t stream)
{
    return run_impl(A, Bc, idx, C, m, n, k, N, M, V, alpha, bias, act, nullptr, 0, kNoTuning, stream, true);
}

extern "C" nmspmm_status_t nmspmm_run_ws(const float *A, const float *Bc, const uint8_t *idx,
                                         float *C, int64_t m, int64_t n, int64_t k, int N, int M,
                                         int V, float alpha, const float *bias, nmspmm_act_t act,
                                         void *workspace, size_t workspace_bytes, hipStream_t stream)
{
    return run_impl(A, Bc, idx, C, m, n, k, N, M, V, alpha, bias, act, workspace, workspace_bytes, kNoTuning,
                    stream, true);
}

extern "C" nmspmm_status_t nmspmm_run_tuned(const float *A, const float *Bc, const uint8_t *idx, float *C,
                                            int64_t m, int64_t n, int64_t k, int N, int M, int V, float alpha,
                                            const float *bias, nmspmm_act_t act, void *workspace,
                                            size_t workspace_bytes, const char *tuning, hipStream_t stream)
{
    Tuning t;
    if (!parse_tuning(tuning, t)) return NMSPMM_ERR_INVALID_ARG;
    return run_impl(A, Bc, idx, C, m, n, k, N, M, V, alpha, bias, act, workspace, workspace_bytes, t, stream);
}

extern "C" int64_t nmspmm_workspace_bytes_tuned(int64_t m, int64_t n, int64_t k, int N, int M, int V,
                                                const char *tuning)
{
    Tuning t;
    if (!parse_tuning(tuning, t) || !shape_ok(m, n, k, N, M, V) || !sizes_fit(m, n, k)) return -1;
    if (m == 0 || n == 0) return 0;
    // buffers aligned as the allocator returns them
    alignas(64) static const float probe[16] = {};
    return plan_ws_bytes(make_ws_plan(probe, probe, probe, m, n, k, N, M, V, t));
}

extern "C" int64_t nmspmm_workspace_bytes(int64_t m, int64_t n, int64_t k, int N, int M, int V)
{
    return nmspmm_workspace_bytes_tuned(m, n, k, N, M, V, nullptr);
}

extern "C" nmspmm_status_t nmspmm_run(const float *A, const float *Bc, const uint8_t *idx,
                                      float *C, int64_t m, int64_t n, int64_t k, int N, int M,
                                      int V, hipStream_t stream)
{
    return nmspmm_run_ex(A, Bc, idx, C, m, n, k, N, M, V, 1.f, nullptr, NMSPMM_ACT_NONE, stream);
}

// ---------------------------------------------------------------------------
// nmspmm_run_noalloc: nmspmm_run_ws with the workspace in a static device
// array instead of caller memory, for callers that cannot allocate.  Every
// device the library runs on holds its own copy of the array (module scope)
// until the process ends; its address on a device is looked up once, on the
// first call there, and the kernels take that address.  Each call rewrites
// every byte of the scratch that its kernels read (the transposed A and the
// gather offsets, or every split's partial tiles), so nothing has to start
// at zero; calls that overlap on one device share the array and race.
// ---------------------------------------------------------------------------
namespace {

static __device__ __align__(256) unsigned char scratch[NMSPMM_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::atomic<void *> g_scratch[kMaxDevices];
std::mutex g_scratch_mu;

// The current device's address of `scratch` (the host-side symbol is only a
// stand-in for it).
hipError_t scratch_on_current_device(void **out)
{
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    void *p = g_scratch[dev].load(std::memory_order_acquire);
    if (!p) {
        std::lock_guard<std::mutex> lock(g_scratch_mu);
        p = g_scratch[dev].load(std::memory_order_relaxed);
        if (!p) {
            e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
            if (e != hipSuccess || !p) return e != hipSuccess ? e : hipErrorInvalidSymbol;
            g_scratch[dev].store(p, std::memory_order_release);
        }
    }
    *out = p;
    return hipSuccess;
}

}  // namespace

extern "C" nmspmm_status_t nmspmm_run_noalloc(const float *A, const float *Bc, const uint8_t *idx, float *C,
                                              int64_t m, int64_t n, int64_t k, int N, int M, int V,
                                              float alpha, const float *bias, nmspmm_act_t act,
                                              hipStream_t stream)
{
    const nmspmm_status_t st = check_run_args(A, Bc, idx, C, m, n, k, N, M, V, bias, act);
    if (st != NMSPMM_OK || m == 0 || n == 0) return st;
    // the workspace the plan of nmspmm_run_ws takes for these buffers
    const int64_t need = plan_ws_bytes(make_ws_plan(A, Bc, C, m, n, k, N, M, V, kNoTuning));
    if (need > (int64_t)NMSPMM_NOALLOC_SCRATCH_BYTES) return NMSPMM_ERR_SCRATCH;
    void *ws = nullptr;
    if (need > 0 && scratch_on_current_device(&ws) != hipSuccess) return NMSPMM_ERR_HIP;
    return run_impl(A, Bc, idx, C, m, n, k, N, M, V, alpha, bias, act, ws,
                    need > 0 ? (size_t)NMSPMM_NOALLOC_SCRATCH_BYTES : 0, kNoTuning, stream);
}

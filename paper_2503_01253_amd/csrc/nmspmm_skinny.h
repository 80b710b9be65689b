// Host-side entry of the streaming kernel for short products (nmspmm_skinny.hip).
#ifndef NMSPMM_SKINNY_H
#define NMSPMM_SKINNY_H

#include <hip/hip_runtime_api.h>

#include <cstdint>

#include "nmspmm_tiled.h"

namespace nmspmm {

struct SkinnyArgs {
    const float *A;
    const float *Bc;
    const uint8_t *idx;
    float *C;
    int64_t m, n, k;
    int N, M, V;
    int splits;          // workgroups per output tile along k (>1: atomic adds into a zeroed C)
    int tiles_m, tiles_n;
    int cw;              // windows per staged chunk of A: cw * M <= skinny_chunk_cols(RT)
    Epilogue epi;        // applied by the stores when splits == 1
    int stream_b;        // 1: Bc loads with the non-temporal hint (Bc much larger than L2)
};

int skinny_rows(int RT);        // rows of C per workgroup with RT row tiles
int skinny_chunk_cols(int RT);  // columns of A per staged chunk with RT row tiles

// RT: row tiles of 16 rows per workgroup (1 or 2); BV: columns per lane per B
// read (1, 2 or 4); QPW: quads per wave per round (1, 2, 4 or 8); COLS:
// columns of C per workgroup (32, 64, 128 or 256).  A must be 16-byte aligned
// and M a multiple of 4 (16-byte loads of A along k).
bool skinny_has(int RT, int BV, int QPW, int COLS);
hipError_t launch_skinny(int RT, int BV, int QPW, int COLS, const SkinnyArgs &a, hipStream_t stream);

}  // namespace nmspmm

#endif

// Host-side entry of the pipelined streaming kernel (nmspmm_stream.hip).
#ifndef NMSPMM_STREAM_H
#define NMSPMM_STREAM_H

#include <hip/hip_runtime_api.h>

#include <cstdint>

#include "nmspmm_tiled.h"

namespace nmspmm {

struct StreamArgs {
    const float *A;
    const float *Bc;
    const uint8_t *idx;
    float *C;
    int64_t m, n, k;
    int N, M, V;
    int splits;          // workgroups per output tile along k (>1: atomic adds into a zeroed C)
    int tiles_m, tiles_n;
    int sw;              // windows per stage: sw * M <= stream_stage_cols(), sw * N <= RB
    Epilogue epi;        // applied by the stores when splits == 1
    float *ws;           // split-k workspace (tiles * splits partial tiles), or null: atomics
};

int stream_rows(int RT);               // rows of C per workgroup
int stream_cols(int BV, int CPW);      // columns of C per workgroup
int stream_stage_cols();               // columns of A per stage (KS)

// RT: row tiles of 16 rows (1, 2 or 4); BV: columns per lane per Bc read (1,
// 2 or 4, with V a multiple of 16 * BV); CPW: column groups per compute wave;
// RB: compressed rows per stage (16, 32 or 64).  A, Bc and C must be 16-byte
// aligned, M a multiple of 4 and at most stream_stage_cols().
bool stream_has(int RT, int BV, int CPW, int RB);
hipError_t launch_stream(int RT, int BV, int CPW, int RB, const StreamArgs &a, hipStream_t stream);

}  // namespace nmspmm

#endif

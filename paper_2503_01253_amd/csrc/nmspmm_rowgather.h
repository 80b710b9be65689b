// Host-side entry of the row-gather kernel for the thinnest products
// (nmspmm_rowgather.hip).
#ifndef NMSPMM_ROWGATHER_H
#define NMSPMM_ROWGATHER_H

#include <hip/hip_runtime_api.h>

#include <cstdint>

#include "nmspmm_tiled.h"

namespace nmspmm {

struct RowGatherArgs {
    const float *A;
    const float *Bc;
    const uint8_t *idx;
    float *C;
    int64_t m, n, k;
    int N, M, V;
    Epilogue epi;
    int stream_b;    // 1: Bc loads with the non-temporal hint (Bc much larger than L2)
};

// A variant: RT row tiles of 16 (at most 16*RT rows), a strip of 16*CT
// columns per workgroup (V a multiple of it), NW waves, D quads in flight per
// wave.
struct RowGatherCfg {
    int RT, CT, NW, D;
};

bool rowgather_has(const RowGatherCfg &c);

// Whether the kernel can run this shape (sizes within its 32-bit offsets).
bool rowgather_fits(const RowGatherCfg &c, int64_t m, int64_t n, int64_t k, int N, int M, int V);

// One launch, no workspace: every output written once.
hipError_t launch_rowgather(const RowGatherCfg &c, const RowGatherArgs &a, hipStream_t stream);

}  // namespace nmspmm

#endif

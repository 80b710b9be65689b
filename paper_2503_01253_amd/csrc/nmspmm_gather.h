// Host-side entry of the direct-gather kernel for short products
// (nmspmm_gather.hip).
#ifndef NMSPMM_GATHER_H
#define NMSPMM_GATHER_H

#include <hip/hip_runtime_api.h>

#include <cstdint>

#include "nmspmm_tiled.h"

namespace nmspmm {

struct GatherArgs {
    const float *A;
    const float *Bc;
    const uint8_t *idx;
    float *C;
    int64_t m, n, k;
    int N, M, V;
    int splits;      // workgroups per column strip along the compressed rows
    int halves;      // row halves (1 or 2, splits == 1 only): each a workgroup of 16*RT rows
    Epilogue epi;    // applied by the stores when splits == 1
    void *ws;        // workspace of gather_layout(...).total bytes, 256-byte aligned
};

// A variant: RT row tiles of 16 (rows 16*RT), CT column tiles of 16 (a strip
// of 16*CT columns per workgroup, CT = 2 or 4), NW waves, D quads in flight
// per wave.
struct GatherCfg {
    int RT, CT, NW, D;
    int H = 1;       // row halves of 16*RT rows each (splits == 1 only)
};

int gather_rows(int RT);  // 16 * RT
bool gather_has(const GatherCfg &c);

// Workspace parts, each starting on a 256-byte boundary:
//   At   : k x gather_rows(RT) floats, A transposed, rows past m zero;
//   off  : (n/V) x w int32, the byte offset into At of the row of A that
//          compressed row u gathers for column block b (at off[b*w + u]);
//   part : splits > 1 only, (n/(16*CT)) x splits partial strips of
//          gather_rows(RT) x 16*CT floats (strip-major, splits consecutive).
struct GatherLayout {
    int64_t at, off, part, total;  // byte offsets of the parts, total size
};
GatherLayout gather_layout(const GatherCfg &c, int64_t n, int64_t k, int N, int M, int V, int splits);

// The transposition and offset pass, then the strip kernel.  With splits > 1
// the partial strips land in the workspace and the caller sums them.
hipError_t launch_gather(const GatherCfg &c, const GatherArgs &a, hipStream_t stream);

}  // namespace nmspmm

#endif

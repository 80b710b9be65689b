// Host-side entry points of the tiled-kernel instantiation units.
#ifndef NMSPMM_TILES_H
#define NMSPMM_TILES_H

#include <hip/hip_runtime_api.h>

namespace nmspmm {

struct TiledArgs;

#define NMSPMM_DECLARE_TILE(name)                                                         \
    hipError_t launch_tiled_##name(int BV, int KA, int NQ, const TiledArgs &a, hipStream_t stream); \
    bool tiled_fits_##name(int BV, int KA, int NQ);

NMSPMM_DECLARE_TILE(256x256)
NMSPMM_DECLARE_TILE(128x512)
NMSPMM_DECLARE_TILE(128x128)
NMSPMM_DECLARE_TILE(64x512)
NMSPMM_DECLARE_TILE(16x512)
NMSPMM_DECLARE_TILE(256x256m32)
NMSPMM_DECLARE_TILE(128x512m32)
NMSPMM_DECLARE_TILE(128x128m32)
NMSPMM_DECLARE_TILE(64x512m32)
NMSPMM_DECLARE_TILE(128x256)
NMSPMM_DECLARE_TILE(256x128)
NMSPMM_DECLARE_TILE(128x256m32)
NMSPMM_DECLARE_TILE(64x1024m32)
NMSPMM_DECLARE_TILE(256x256m32w16)
NMSPMM_DECLARE_TILE(128x512m32w16)
NMSPMM_DECLARE_TILE(128x256m32w16)

#undef NMSPMM_DECLARE_TILE

}  // namespace nmspmm

#endif

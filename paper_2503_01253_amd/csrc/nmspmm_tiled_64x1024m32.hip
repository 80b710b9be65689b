// Instantiations of the tiled kernel for 64 x 1024 tiles on the 32x32x2 fp32
// MFMA, 1 x 8 waves of 64 x 128 (all column-group widths and stage
// shapes that fit in LDS).
#include "nmspmm_tiled.h"
#include "nmspmm_tiles.h"

namespace nmspmm {

using Tile_64x1024m32 = TileCfg<64, 1024, 64, 128, 32>;

hipError_t launch_tiled_64x1024m32(int BV, int KA, int NQ, const TiledArgs &a, hipStream_t stream)
{
    return launch_tiled_any<Tile_64x1024m32>(BV, KA, NQ, a, stream);
}

bool tiled_fits_64x1024m32(int BV, int KA, int NQ) { return tiled_fits<Tile_64x1024m32>(BV, KA, NQ); }

}  // namespace nmspmm

// Instantiations of the tiled kernel for 256 x 128 tiles on the 16x16x4 fp32
// MFMA, 4 x 2 waves of 64 x 64 (all column-group widths and stage
// shapes that fit in LDS).
#include "nmspmm_tiled.h"
#include "nmspmm_tiles.h"

namespace nmspmm {

using Tile_256x128 = TileCfg<256, 128, 64, 64>;

hipError_t launch_tiled_256x128(int BV, int KA, int NQ, const TiledArgs &a, hipStream_t stream)
{
    return launch_tiled_any<Tile_256x128>(BV, KA, NQ, a, stream);
}

bool tiled_fits_256x128(int BV, int KA, int NQ) { return tiled_fits<Tile_256x128>(BV, KA, NQ); }

}  // namespace nmspmm

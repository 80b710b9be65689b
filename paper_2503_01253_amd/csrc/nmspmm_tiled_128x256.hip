// Instantiations of the tiled kernel for 128 x 256 tiles on the 16x16x4 fp32
// MFMA, 2 x 4 waves of 64 x 64 (all column-group widths and stage
// shapes that fit in LDS).
#include "nmspmm_tiled.h"
#include "nmspmm_tiles.h"

namespace nmspmm {

using Tile_128x256 = TileCfg<128, 256, 64, 64>;

hipError_t launch_tiled_128x256(int BV, int KA, int NQ, const TiledArgs &a, hipStream_t stream)
{
    return launch_tiled_any<Tile_128x256>(BV, KA, NQ, a, stream);
}

bool tiled_fits_128x256(int BV, int KA, int NQ) { return tiled_fits<Tile_128x256>(BV, KA, NQ); }

}  // namespace nmspmm

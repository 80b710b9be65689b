// Instantiations of the tiled kernel for 256 x 256 tiles (all column-group
// widths and stage shapes that fit in LDS).
#include "nmspmm_tiled.h"
#include "nmspmm_tiles.h"

namespace nmspmm {

using Tile_256x256 = TileCfg<256, 256, 128, 64>;

hipError_t launch_tiled_256x256(int BV, int KA, int NQ, const TiledArgs &a, hipStream_t stream)
{
    return launch_tiled_any<Tile_256x256>(BV, KA, NQ, a, stream);
}

bool tiled_fits_256x256(int BV, int KA, int NQ) { return tiled_fits<Tile_256x256>(BV, KA, NQ); }

}  // namespace nmspmm

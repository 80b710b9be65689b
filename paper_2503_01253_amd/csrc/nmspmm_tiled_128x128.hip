// Instantiations of the tiled kernel for 128 x 128 tiles (all column-group
// widths and stage shapes that fit in LDS).
#include "nmspmm_tiled.h"
#include "nmspmm_tiles.h"

namespace nmspmm {

using Tile_128x128 = TileCfg<128, 128, 64, 64>;

hipError_t launch_tiled_128x128(int BV, int KA, int NQ, const TiledArgs &a, hipStream_t stream)
{
    return launch_tiled_any<Tile_128x128>(BV, KA, NQ, a, stream);
}

bool tiled_fits_128x128(int BV, int KA, int NQ) { return tiled_fits<Tile_128x128>(BV, KA, NQ); }

}  // namespace nmspmm

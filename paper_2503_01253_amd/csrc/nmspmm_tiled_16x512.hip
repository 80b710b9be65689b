// Instantiations of the tiled kernel for 16 x 512 tiles (all column-group
// widths and stage shapes that fit in LDS).
#include "nmspmm_tiled.h"
#include "nmspmm_tiles.h"

namespace nmspmm {

using Tile_16x512 = TileCfg<16, 512, 16, 64>;

hipError_t launch_tiled_16x512(int BV, int KA, int NQ, const TiledArgs &a, hipStream_t stream)
{
    return launch_tiled_any<Tile_16x512>(BV, KA, NQ, a, stream);
}

bool tiled_fits_16x512(int BV, int KA, int NQ) { return tiled_fits<Tile_16x512>(BV, KA, NQ); }

}  // namespace nmspmm

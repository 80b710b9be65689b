// Instantiations of the tiled kernel for 128x512 tiles with sixteen 64 x 64
// wave tiles (four waves per SIMD; all column-group widths and stage shapes
// that fit in LDS).
#include "nmspmm_tiled.h"
#include "nmspmm_tiles.h"

namespace nmspmm {

using Tile_128x512w16 = TileCfg<128, 512, 64, 64>;

hipError_t launch_tiled_128x512w16(int BV, int KA, int NQ, const TiledArgs &a, hipStream_t stream)
{
    return launch_tiled_any<Tile_128x512w16>(BV, KA, NQ, a, stream);
}

bool tiled_fits_128x512w16(int BV, int KA, int NQ) { return tiled_fits<Tile_128x512w16>(BV, KA, NQ); }

}  // namespace nmspmm

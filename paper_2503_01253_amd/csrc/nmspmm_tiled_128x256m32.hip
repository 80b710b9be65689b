// Instantiations of the tiled kernel for 128 x 256 tiles on the 32x32x2 fp32
// MFMA, 1 x 8 waves of 128 x 32 (all column-group widths and stage
// shapes that fit in LDS).
#include "nmspmm_tiled.h"
#include "nmspmm_tiles.h"

namespace nmspmm {

using Tile_128x256m32 = TileCfg<128, 256, 128, 32, 32>;

hipError_t launch_tiled_128x256m32(int BV, int KA, int NQ, const TiledArgs &a, hipStream_t stream)
{
    return launch_tiled_any<Tile_128x256m32>(BV, KA, NQ, a, stream);
}

bool tiled_fits_128x256m32(int BV, int KA, int NQ) { return tiled_fits<Tile_128x256m32>(BV, KA, NQ); }

}  // namespace nmspmm

// Instantiations of the tiled kernel for 128 x 512 tiles on the 32x32x2 fp32
// MFMA, 1 x 16 waves of 128 x 32
// (16 waves, four per SIMD: while some wait on their loads the others keep the
// matrix pipe busy; 64 or fewer accumulators per lane fit the 128 VGPRs).
#include "nmspmm_tiled.h"
#include "nmspmm_tiles.h"

namespace nmspmm {

using Tile_128x512m32w16 = TileCfg<128, 512, 128, 32, 32>;

hipError_t launch_tiled_128x512m32w16(int BV, int KA, int NQ, const TiledArgs &a, hipStream_t stream)
{
    return launch_tiled_any<Tile_128x512m32w16>(BV, KA, NQ, a, stream);
}

bool tiled_fits_128x512m32w16(int BV, int KA, int NQ) { return tiled_fits<Tile_128x512m32w16>(BV, KA, NQ); }

}  // namespace nmspmm

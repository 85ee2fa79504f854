// gemm_mx_11n.hip -- the one-chunk, groups-of-16 BFP GEMM on the smaller
// tiles (256x128, 256x64, 128x64, 128x128) that the dispatch picks for narrow or small
// GEMMs; compiled on its own so that it builds in parallel with the rest.
#include "gemm_mx.h"

namespace fastbfp {

#define FASTBFP_MX11_TILES(FA, FB)                   \
  FASTBFP_MX11_TILE_INSTANTIATE(256, 128, FA, FB)   \
  FASTBFP_MX11_TILE_INSTANTIATE(256, 64, FA, FB)    \
  FASTBFP_MX11_TILE_INSTANTIATE(128, 64, FA, FB)    \
  FASTBFP_MX11_TILE_INSTANTIATE(128, 128, FA, FB)

FASTBFP_MX11_TILES(0, 0)
FASTBFP_MX11_TILES(0, 1)
FASTBFP_MX11_TILES(1, 0)
FASTBFP_MX11_TILES(1, 1)

}  // namespace fastbfp

// gemm_mx_11n_01.hip -- the one-chunk, groups-of-16 BFP GEMM on the smaller
// tiles (256x128, 256x64, 128x64, 128x128) that the dispatch picks for narrow
// or small GEMMs, with A / B planes of FP4 codes = 0 / 1; FP32 or converted
// output.  One file per operand-format pair so that they build in parallel.
#include "gemm_mx.h"

namespace fastbfp {

FASTBFP_MX11_TILE_INSTANTIATE(256, 128, 0, 1)
FASTBFP_MX11_TILE_INSTANTIATE(256, 64, 0, 1)
FASTBFP_MX11_TILE_INSTANTIATE(128, 64, 0, 1)
FASTBFP_MX11_TILE_INSTANTIATE(128, 128, 0, 1)

}  // namespace fastbfp

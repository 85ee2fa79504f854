// gemm_mx_22_g32.hip -- the BFP GEMM with 2 chunk plane(s) of A and 2 of B, groups of
// 32, every plane-0 format (FP6 or FP4 codes) of either operand.
#include "gemm_mx.h"

namespace fastbfp {

FASTBFP_MX_INSTANTIATE(2, 2, 0, 0, 32)
FASTBFP_MX_INSTANTIATE(2, 2, 0, 1, 32)
FASTBFP_MX_INSTANTIATE(2, 2, 1, 0, 32)
FASTBFP_MX_INSTANTIATE(2, 2, 1, 1, 32)

}  // namespace fastbfp

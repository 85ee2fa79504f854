// gemm_mx_21.hip -- the BFP GEMM with 2 chunk plane(s) of A and 1 of B, groups of
// 16, every plane-0 format (FP6 or FP4 codes) of either operand.
#include "gemm_mx.h"

namespace fastbfp {

FASTBFP_MX_INSTANTIATE(2, 1, 0, 0, 16)
FASTBFP_MX_INSTANTIATE(2, 1, 0, 1, 16)
FASTBFP_MX_INSTANTIATE(2, 1, 1, 0, 16)
FASTBFP_MX_INSTANTIATE(2, 1, 1, 1, 16)

}  // namespace fastbfp

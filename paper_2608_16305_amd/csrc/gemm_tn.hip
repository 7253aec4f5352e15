// Weight-gradient products dW = dy^T x (both operands contiguous along the output dimensions): this layout's instances of the strip GEMM.
#include "gemm.h"

namespace mtgnn {

MTGNN_GEMM_INSTANCES_TN()

}  // namespace mtgnn

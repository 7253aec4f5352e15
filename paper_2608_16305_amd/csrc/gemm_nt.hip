// Forward products y = x W^T (both operands contiguous along k): this layout's instances of the strip GEMM.
#include "gemm.h"

namespace mtgnn {

MTGNN_GEMM_INSTANCES()

}  // namespace mtgnn

// Data-gradient products dx = dy W (A contiguous along k, B along the output columns): this layout's instances of the strip GEMM.
#include "gemm.h"

namespace mtgnn {

MTGNN_GEMM_INSTANCES_NN()

}  // namespace mtgnn

// Weight-gradient products dW = dy^T x (both operands contiguous along the output dimensions).
#include "gemm.h"

namespace mtgnn {

template <class Site, bool AK, bool BK>
mtgnn_status gemm_launch(const GemmArgs& g, int dtype_a, int dtype_b, int ksplit, hipStream_t s) {
  return gemm_launch_impl<Site, AK, BK>(g, dtype_a, dtype_b, ksplit, s);
}

template <class Site, bool AK, bool BK>
mtgnn_status gemm_batch_launch(const GemmArgs* gs, int n, int zper, int dtype_a, int dtype_b, hipStream_t s) {
  return gemm_batch_launch_impl<Site, AK, BK>(gs, n, zper, dtype_a, dtype_b, s);
}

template mtgnn_status gemm_launch<site::Generic, false, false>(const GemmArgs&, int, int, int, hipStream_t);
template mtgnn_status gemm_launch<site::KvDw, false, false>(const GemmArgs&, int, int, int, hipStream_t);

template mtgnn_status gemm_batch_launch<site::Generic, false, false>(const GemmArgs*, int, int, int, int, hipStream_t);
template mtgnn_status gemm_batch_launch<site::GruDw, false, false>(const GemmArgs*, int, int, int, int, hipStream_t);

}  // namespace mtgnn

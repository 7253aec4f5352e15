// Host side of the weight-stationary product (gemm_rs.h).
#include "gemm_rs.h"

namespace mtgnn {

namespace {

int cu_count() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  static int cache[64] = {0};   // per device; every writer stores the same value
  if (cache[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    cache[dev] = n;
  }
  return cache[dev];
}

}  // namespace

bool gemm_rs_applicable(const GemmArgs& g) {
  const int64_t nct = cdiv(g.N, 16), kc = cdiv(g.K, 16);
  return g.M > 0 && nct == 13 && (kc == 13 || kc == 14) && ((uintptr_t)g.A % 16) == 0 && g.a_sk == 1 &&
         g.a_si % 4 == 0 && g.K % 4 == 0 && g.K_dev == nullptr && g.ones_col < 0 && g.c_split_stride == 0 &&
         !g.accumulate && !g.relu && g.gate == nullptr && !g.round_bf16 && g.tg_part == nullptr && cu_count() > 0;
}

mtgnn_status gemm_rs_launch(const GemmArgs& g0, hipStream_t s) {
  GemmArgs g = g0;
  g.b_vec = (g.b_sk == 1 && vec_ok(g.B, g.b_sj, sizeof(float))) ? 1 : 0;
  const int64_t tiles = cdiv(g.M, 16);
  const unsigned grid = (unsigned)(tiles < cu_count() ? tiles : cu_count());
  if (cdiv(g.K, 16) == 13) k_gemm_rs<site::KvProj, 13, 13, 1><<<grid, G_THREADS, 0, s>>>(g);
  else k_gemm_rs<site::KvProj, 13, 14, 1><<<grid, G_THREADS, 0, s>>>(g);
  MTGNN_CHECK_LAUNCH("gemm_rs");
  return MTGNN_OK;
}

}  // namespace mtgnn

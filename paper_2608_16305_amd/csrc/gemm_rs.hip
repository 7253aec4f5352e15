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

mtgnn_status gemm_rs_launch(const GemmArgs& g0, hipStream_t s, bool bf16_weights) {
  GemmArgs g = g0;
  g.b_vec = (!bf16_weights && g.b_sk == 1 && vec_ok(g.B, g.b_sj, sizeof(float))) ? 1 : 0;
  const int64_t tiles = cdiv(g.M, 16);
  const unsigned grid = (unsigned)(tiles < cu_count() ? tiles : cu_count());
  if (bf16_weights) {
    if (cdiv(g.K, 16) == 13) k_gemm_rs<site::KvProj, 13, 13, 1, uint16_t><<<grid, G_THREADS, 0, s>>>(g);
    else k_gemm_rs<site::KvProj, 13, 14, 1, uint16_t><<<grid, G_THREADS, 0, s>>>(g);
  } else if (cdiv(g.K, 16) == 13) {
    k_gemm_rs<site::KvProj, 13, 13, 1><<<grid, G_THREADS, 0, s>>>(g);
  } else {
    k_gemm_rs<site::KvProj, 13, 14, 1><<<grid, G_THREADS, 0, s>>>(g);
  }
  MTGNN_CHECK_LAUNCH("gemm_rs");
  return MTGNN_OK;
}

}  // namespace mtgnn

namespace mtgnn {

namespace {
constexpr int DW_RS_MAX_BLOCKS = 256;   // partials the workspace is sized for (one per CU of an MI355X)
}

bool dw_rs_applicable(const float* X, int64_t ldx, int nx, const void* Y, int y_dtype, int64_t ldy, int ny) {
  const int nj = (int)cdiv(ny + 1, 16);
  return y_dtype == MTGNN_F32 && nx > 192 && nx <= 208 && nx % 4 == 0 && ny % 4 == 0 && (nj == 13 || nj == 14) &&
         ((uintptr_t)X % 16) == 0 && ((uintptr_t)Y % 16) == 0 && ldx % 4 == 0 && ldy % 4 == 0 && cu_count() > 0;
}

size_t dw_rs_ws_bytes(int nx, int ny) { return sizeof(float) * (size_t)DW_RS_MAX_BLOCKS * nx * (ny + 1); }

mtgnn_status dw_rs_launch(const float* X, int64_t ldx, int nx, const float* Y, int64_t ldy, int ny, int64_t R,
                          const int32_t* R_dev, float* dW, int64_t lddw, float* db, void* ws, size_t ws_bytes,
                          hipStream_t s) {
  return dw_rs_launch_rows2(X, ldx, nx, Y, ldy, ny, R, R_dev, dW, nullptr, lddw, db, nullptr, nx, ws, ws_bytes, s);
}

mtgnn_status dw_rs_launch_rows2(const float* X, int64_t ldx, int nx, const float* Y, int64_t ldy, int ny, int64_t R,
                                const int32_t* R_dev, float* dW, float* dW_hi, int64_t lddw, float* db, float* db_hi,
                                int row_split, void* ws, size_t ws_bytes, hipStream_t s) {
  const size_t per = sizeof(float) * (size_t)nx * (ny + 1);
  int64_t grid = cu_count();
  if ((int64_t)(ws_bytes / per) < grid) grid = (int64_t)(ws_bytes / per);
  if (grid < 1) return MTGNN_EWORKSPACE;
  float* part = (float*)ws;
  {
    TimedScope ts(site::KvDw::name, s);
    if (cdiv(ny + 1, 16) == 13)
      k_dw_rs<site::KvDw, 13><<<(unsigned)grid, G_THREADS, 0, s>>>(X, ldx, nx, Y, ldy, ny, R, R_dev, part);
    else
      k_dw_rs<site::KvDw, 14><<<(unsigned)grid, G_THREADS, 0, s>>>(X, ldx, nx, Y, ldy, ny, R, R_dev, part);
  }
  MTGNN_CHECK_LAUNCH("dw_rs");
  const int64_t outs = (int64_t)nx * (ny + 1);
  if (dW_hi)
    k_splitk_reduce_rows2<<<(unsigned)cdiv(outs, 64), 256, 0, s>>>(part, outs, (int)grid, nx, ny + 1, dW, dW_hi, lddw,
                                                                  ny, db, db_hi, row_split);
  else
    k_splitk_reduce<<<(unsigned)cdiv(outs, 64), 256, 0, s>>>(part, outs, (int)grid, nx, ny + 1, dW, lddw, ny, db);
  MTGNN_CHECK_LAUNCH("splitk_reduce");
  return MTGNN_OK;
}

int dw_os_cu_count() { return cu_count(); }

template <class Site>
mtgnn_status dw_os_launch(const DwOsBatch& b, int grid, hipStream_t s) {
  {
    TimedScope ts("dw_os", s);
    k_dw_os<Site><<<(unsigned)grid, G_THREADS, 0, s>>>(b);
  }
  MTGNN_CHECK_LAUNCH("dw_os");
  return MTGNN_OK;
}

template mtgnn_status dw_os_launch<site::Generic>(const DwOsBatch&, int, hipStream_t);
template mtgnn_status dw_os_launch<site::GruDw>(const DwOsBatch&, int, hipStream_t);

}  // namespace mtgnn

// Split-K reduction and launch-shape helpers of the strip GEMM.
#include "gemm.h"

namespace mtgnn {

// 64 outputs per block; the 4 waves sum interleaved split slices, combined in a fixed order.
__global__ __launch_bounds__(256) void k_splitk_reduce(const float* __restrict__ part, int64_t split_stride,
                                                       int nsplit, int64_t rows, int64_t cols, float* __restrict__ out,
                                                       int64_t ldo, int64_t ones_col, float* __restrict__ col_out) {
  __shared__ float red[4][64];
  const int64_t e = (int64_t)blockIdx.x * 64 + (threadIdx.x & 63);
  const int g = threadIdx.x >> 6;
  float s = 0.f;
  if (e < rows * cols) {
    int z = g;
    for (; z + 12 < nsplit; z += 16) {   // four loads in flight
      const float a0 = part[(int64_t)z * split_stride + e], a1 = part[(int64_t)(z + 4) * split_stride + e];
      const float a2 = part[(int64_t)(z + 8) * split_stride + e], a3 = part[(int64_t)(z + 12) * split_stride + e];
      s += ((a0 + a1) + a2) + a3;
    }
    for (; z < nsplit; z += 4) s += part[(int64_t)z * split_stride + e];
  }
  red[g][threadIdx.x & 63] = s;
  __syncthreads();
  if (g != 0 || e >= rows * cols) return;
  const int l = threadIdx.x;
  s = ((red[0][l] + red[1][l]) + red[2][l]) + red[3][l];
  const int64_t i = e / cols, j = e % cols;
  if (j == ones_col) col_out[i] = s;
  else out[i * ldo + j] = s;
}

int gemm_strip_width(int64_t N) {
  static const int widths[] = {64, 128, 160, 208, 256};
  const int64_t strips = cdiv(N, 256);
  const int64_t per = cdiv(N, strips);
  for (int w : widths)
    if (w >= per) return w;
  return 256;
}

int gemm_tile_width(int64_t M, int64_t N, int ksplit) {
  const int full = gemm_strip_width(N);
  const int64_t blocks = cdiv(M, 64 * G_WM) * cdiv(N, full) * (ksplit < 1 ? 1 : ksplit);
  return blocks < 1024 ? 64 : full;
}

// Up to 16 K reduction rows, 64 x 64 tiles over 128-row chunks (each block one
// short reduction; the grid is tiles x chunks).  Larger reductions keep full
// strips and cut the rows into chunks of >= 256 so the grid has about 1536
// blocks at the host row maximum (device-side counts often leave fewer active).
DwPlan dw_plan(int64_t R, int64_t N, int64_t K) {
  DwPlan p;
  const int64_t r = R < 1 ? 1 : R;
  if (r <= 16384) {
    p.bn = 64;
    p.bk = 64;
    p.kchunk = 128;
  } else {
    p.bn = gemm_strip_width(K);
    p.bk = G_BK;
    const int64_t tiles = cdiv(N, 64 * G_WM) * cdiv(K, p.bn);
    int64_t want = cdiv(1536, tiles);
    if (want > 512) want = 512;
    if (want < 1) want = 1;
    p.kchunk = cdiv(cdiv(r, want), G_BK) * G_BK;
    if (p.kchunk < 256) p.kchunk = 256;
  }
  p.ksplit = (int)cdiv(r, p.kchunk);
  if (p.ksplit == 1) p.kchunk = r;
  return p;
}

size_t linear_dw_ws_bytes(int64_t R, int64_t N, int64_t K) {
  const DwPlan p = dw_plan(R, N, K + 1);
  return p.ksplit > 1 ? sizeof(float) * (size_t)p.ksplit * N * (K + 1) : 0;
}

}  // namespace mtgnn

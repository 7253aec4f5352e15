// Host launchers for the strided MFMA GEMM and its split-K reduction.
#include "gemm.h"

namespace mtgnn {

__global__ void k_splitk_reduce(const float* __restrict__ part, int64_t split_stride, int nsplit, int64_t rows,
                                int64_t cols, float* __restrict__ out, int64_t ldo, int accumulate) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= rows * cols) return;
  const int64_t i = e / cols, j = e % cols;
  float s = 0.f;
  for (int z = 0; z < nsplit; ++z) s += part[(int64_t)z * split_stride + e];
  out[i * ldo + j] = accumulate ? out[i * ldo + j] + s : s;
}

namespace {

template <typename TA, typename TB>
mtgnn_status launch4(const GemmArgs& g, bool ak, bool bk, dim3 grid, hipStream_t s) {
  if (ak && bk) k_gemm_f32<TA, TB, true, true><<<grid, G_THREADS, 0, s>>>(g);
  else if (ak && !bk) k_gemm_f32<TA, TB, true, false><<<grid, G_THREADS, 0, s>>>(g);
  else if (!ak && bk) k_gemm_f32<TA, TB, false, true><<<grid, G_THREADS, 0, s>>>(g);
  else k_gemm_f32<TA, TB, false, false><<<grid, G_THREADS, 0, s>>>(g);
  MTGNN_CHECK_LAUNCH("gemm");
  return MTGNN_OK;
}

}  // namespace

mtgnn_status gemm_launch(const GemmArgs& g, int dtype_a, int dtype_b, bool a_kcontig, bool b_kcontig, int ksplit,
                         hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return MTGNN_OK;
  dim3 grid((unsigned)cdiv(g.M, G_BM), (unsigned)cdiv(g.N, G_BN), (unsigned)(ksplit < 1 ? 1 : ksplit));
  if (dtype_a == MTGNN_F32 && dtype_b == MTGNN_F32) return launch4<float, float>(g, a_kcontig, b_kcontig, grid, s);
  if (dtype_a == MTGNN_F32 && dtype_b == MTGNN_BF16) return launch4<float, uint16_t>(g, a_kcontig, b_kcontig, grid, s);
  if (dtype_a == MTGNN_BF16 && dtype_b == MTGNN_F32) return launch4<uint16_t, float>(g, a_kcontig, b_kcontig, grid, s);
  return launch4<uint16_t, uint16_t>(g, a_kcontig, b_kcontig, grid, s);
}

mtgnn_status linear_fwd(const void* x, int x_dtype, int64_t ldx, const void* W, int w_dtype, int64_t ldw,
                        const float* bias, float* y, int64_t ldy, int64_t M, const int32_t* M_dev, int64_t N,
                        int64_t K, bool accumulate, hipStream_t s, float* pre_relu, int64_t ldpre, bool round_bf16) {
  GemmArgs g{};
  g.M = M; g.N = N; g.K = K; g.M_dev = M_dev;
  g.A = x; g.a_si = ldx; g.a_sk = 1;
  g.B = W; g.b_sk = 1; g.b_sj = ldw;
  g.C = y; g.ldc = ldy; g.bias = bias; g.accumulate = accumulate ? 1 : 0;
  g.relu = pre_relu ? 1 : 0; g.C2 = pre_relu; g.ldc2 = ldpre;
  g.kchunk = K; g.c_split_stride = 0; g.round_bf16 = round_bf16 ? 1 : 0;
  return gemm_launch(g, x_dtype, w_dtype, true, true, 1, s);
}

mtgnn_status linear_dx(const float* dy, int64_t lddy, const void* W, int w_dtype, int64_t ldw, float* dx,
                       int64_t lddx, int64_t M, const int32_t* M_dev, int64_t N, int64_t K, bool accumulate,
                       hipStream_t s, const float* gate, int64_t ldgate) {
  GemmArgs g{};
  g.M = M; g.N = K; g.K = N; g.M_dev = M_dev;
  g.A = dy; g.a_si = lddy; g.a_sk = 1;
  g.B = W; g.b_sk = ldw; g.b_sj = 1;
  g.C = dx; g.ldc = lddx; g.accumulate = accumulate ? 1 : 0;
  g.kchunk = N; g.c_split_stride = 0; g.gate = gate; g.ldgate = ldgate;
  return gemm_launch(g, MTGNN_F32, w_dtype, true, false, 1, s);
}

namespace {
void dw_split(int64_t R, int64_t N, int64_t K, int& ksplit, int64_t& kchunk) {
  const int64_t tiles = cdiv(N, G_BM) * cdiv(K, G_BN);
  int64_t want = cdiv(1024, tiles);
  int64_t maxs = cdiv(R < 1 ? 1 : R, 512);
  if (want > maxs) want = maxs;
  if (want < 1) want = 1;
  if (want > 256) want = 256;
  kchunk = cdiv(cdiv(R < 1 ? 1 : R, want), G_BK) * G_BK;
  ksplit = (int)cdiv(R < 1 ? 1 : R, kchunk);
}
}  // namespace

size_t linear_dw_ws_bytes(int64_t R, int64_t N, int64_t K) {
  int ks;
  int64_t kc;
  dw_split(R, N, K, ks, kc);
  return ks > 1 ? sizeof(float) * (size_t)ks * N * K : 0;
}

mtgnn_status linear_dw(const float* dy, int64_t lddy, const void* x, int x_dtype, int64_t ldx, float* dW,
                       int64_t lddw, int64_t R, const int32_t* R_dev, int64_t N, int64_t K, void* ws,
                       size_t ws_bytes, hipStream_t s) {
  int ksplit;
  int64_t kchunk;
  dw_split(R, N, K, ksplit, kchunk);
  GemmArgs g{};
  g.M = N; g.N = K; g.K = R; g.K_dev = R_dev;
  g.A = dy; g.a_si = 1; g.a_sk = lddy;
  g.B = x; g.b_sk = ldx; g.b_sj = 1;
  g.kchunk = kchunk;
  if (ksplit == 1) {
    g.C = dW; g.ldc = lddw; g.c_split_stride = 0;
    return gemm_launch(g, MTGNN_F32, x_dtype, false, false, 1, s);
  }
  if (ws_bytes < linear_dw_ws_bytes(R, N, K)) return MTGNN_EWORKSPACE;
  g.C = (float*)ws; g.ldc = K; g.c_split_stride = N * K;
  MTGNN_TRY(gemm_launch(g, MTGNN_F32, x_dtype, false, false, ksplit, s));
  const int64_t tot = N * K;
  k_splitk_reduce<<<(unsigned)cdiv(tot, 256), 256, 0, s>>>((const float*)ws, N * K, ksplit, N, K, dW, lddw, 0);
  MTGNN_CHECK_LAUNCH("splitk_reduce");
  return MTGNN_OK;
}

}  // namespace mtgnn

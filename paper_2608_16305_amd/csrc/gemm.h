// Strided fp32-accumulating MFMA GEMM for gfx950:  C(i,j) = sum_k A(i,k) B(k,j).
//
// A(i,k) = A[i*a_si + k*a_sk], B(k,j) = B[k*b_sk + j*b_sj], C row-major.
// One template covers the three products of a linear layer y = x W^T + b:
//   forward   y  = x  W^T : A = x (k-contiguous),      B(k,j) = W[j][k] (k-contiguous)
//   data grad dx = dy W   : A = dy (k-contiguous),     B(k,j) = W[k][j] (j-contiguous)
//   weight    dW = dy^T x : A(i,k) = dy[k][i] (i-contig.), B(k,j) = x[k][j] (j-contiguous)
// The contiguous dimension of each operand picks the global->LDS load mapping
// (coalesced along it) and an LDS layout whose MFMA fragment reads are
// bank-conflict free.  Inputs may be float32 or bfloat16 (converted on load);
// the MFMA is v_mfma_f32_16x16x4_f32 (lane l supplies A[l%16][l/16] and
// B[l/16][l%16]; accumulator register r of lane l is C[4*(l/16)+r][l%16]).
#pragma once

#include "common.h"

namespace mtgnn {

typedef float f32x4 __attribute__((ext_vector_type(4)));

struct GemmArgs {
  int64_t M, N, K;
  const int32_t* M_dev;        // optional device count clamping M
  const int32_t* K_dev;        // optional device count clamping K
  const void* A;
  int64_t a_si, a_sk;
  const void* B;
  int64_t b_sk, b_sj;
  float* C;
  int64_t ldc;
  const float* bias;           // per output column, or null
  int accumulate;              // C += result
  int relu;                    // write relu(result) to C and the pre-activation to C2
  float* C2;
  int64_t ldc2;
  int64_t kchunk;              // split-K chunk (blockIdx.z covers [z*kchunk, (z+1)*kchunk))
  int64_t c_split_stride;      // element offset of split z's output
  const float* gate;           // optional: result *= (gate(i,j) > 0)  (ReLU backward)
  int64_t ldgate;
  int round_bf16;              // round the stored result to bfloat16 (kept as float32)
};

// Epilogue rounding of a float32 value to the nearest bfloat16 (ties to even), widened back.
__device__ __forceinline__ float round_to_bf16(float v) { return bf16_to_f32(f32_to_bf16(v)); }

constexpr int G_BM = 64, G_BN = 64, G_BK = 16, G_THREADS = 256;

template <bool KCONTIG, int BMN>
struct TileLayout;
// k-contiguous operand: [BMN][BK+1] (row = m or n)
template <int BMN>
struct TileLayout<true, BMN> {
  static constexpr int SIZE = BMN * (G_BK + 1);
  __device__ __forceinline__ static int idx(int mn, int k) { return mn * (G_BK + 1) + k; }
  __device__ __forceinline__ static void coord(int e, int& mn, int& k) { k = e % G_BK; mn = e / G_BK; }
};
// m/n-contiguous operand: [BK][BMN+16]
template <int BMN>
struct TileLayout<false, BMN> {
  static constexpr int SIZE = G_BK * (BMN + 16);
  __device__ __forceinline__ static int idx(int mn, int k) { return k * (BMN + 16) + mn; }
  __device__ __forceinline__ static void coord(int e, int& mn, int& k) { mn = e % BMN; k = e / BMN; }
};

template <typename TA, typename TB, bool A_KCONTIG, bool B_KCONTIG>
__global__ __launch_bounds__(G_THREADS) void k_gemm_f32(GemmArgs g) {
  using LA = TileLayout<A_KCONTIG, G_BM>;
  using LB = TileLayout<B_KCONTIG, G_BN>;
  __shared__ float As[LA::SIZE];
  __shared__ float Bs[LB::SIZE];

  const int64_t M = eff_count(g.M, g.M_dev);
  const int64_t Kall = eff_count(g.K, g.K_dev);
  const int64_t row0 = (int64_t)blockIdx.x * G_BM;
  const int64_t col0 = (int64_t)blockIdx.y * G_BN;
  if (row0 >= M) return;
  const int64_t kbeg = (int64_t)blockIdx.z * g.kchunk;
  const int64_t kend = min(Kall, kbeg + g.kchunk);

  const TA* A = (const TA*)g.A;
  const TB* B = (const TB*)g.B;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int wm = wid >> 1, wn = wid & 1;

  f32x4 acc[2][2];
  for (int i = 0; i < 2; ++i)
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  constexpr int PER_T = (G_BM * G_BK) / G_THREADS;   // 4 elements of A and of B per thread
  float ra[PER_T], rb[PER_T];

  auto load = [&](int64_t k0) {
#pragma unroll
    for (int p = 0; p < PER_T; ++p) {
      int e = tid + p * G_THREADS, mn, k;
      LA::coord(e, mn, k);
      int64_t gi = row0 + mn, gk = k0 + k;
      ra[p] = (gi < M && gk < kend) ? Elem<TA>::load(A, gi * g.a_si + gk * g.a_sk) : 0.f;
      LB::coord(e, mn, k);
      int64_t gj = col0 + mn;
      gk = k0 + k;
      rb[p] = (gj < g.N && gk < kend) ? Elem<TB>::load(B, gk * g.b_sk + gj * g.b_sj) : 0.f;
    }
  };
  auto stash = [&]() {
#pragma unroll
    for (int p = 0; p < PER_T; ++p) {
      int e = tid + p * G_THREADS, mn, k;
      LA::coord(e, mn, k);
      As[LA::idx(mn, k)] = ra[p];
      LB::coord(e, mn, k);
      Bs[LB::idx(mn, k)] = rb[p];
    }
  };

  if (kbeg < kend) {
    load(kbeg);
    for (int64_t k0 = kbeg; k0 < kend; k0 += G_BK) {
      __syncthreads();
      stash();
      __syncthreads();
      if (k0 + G_BK < kend) load(k0 + G_BK);
#pragma unroll
      for (int ks = 0; ks < G_BK; ks += 4) {
        float a[2], b[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) a[i] = As[LA::idx(wm * 32 + i * 16 + (lane & 15), ks + (lane >> 4))];
#pragma unroll
        for (int j = 0; j < 2; ++j) b[j] = Bs[LB::idx(wn * 32 + j * 16 + (lane & 15), ks + (lane >> 4))];
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[j], acc[i][j], 0, 0, 0);
      }
    }
  }

  float* C = g.C + (int64_t)blockIdx.z * g.c_split_stride;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int64_t gj = col0 + wn * 32 + j * 16 + (lane & 15);
      if (gj >= g.N) continue;
      const float bj = g.bias ? g.bias[gj] : 0.f;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t gi = row0 + wm * 32 + i * 16 + 4 * (lane >> 4) + r;
        if (gi >= M) continue;
        float v = acc[i][j][r] + bj;
        if (g.accumulate) v += C[gi * g.ldc + gj];
        if (g.gate && !(g.gate[gi * g.ldgate + gj] > 0.f)) v = 0.f;
        if (g.relu) {
          g.C2[gi * g.ldc2 + gj] = v;
          v = fmaxf(v, 0.f);
        }
        if (g.round_bf16) v = round_to_bf16(v);
        C[gi * g.ldc + gj] = v;
      }
    }
}

// Sums split-K partials in a fixed order: out(i,j) (+)= sum_z part[z](i,j).
__global__ void k_splitk_reduce(const float* __restrict__ part, int64_t split_stride, int nsplit, int64_t rows,
                                int64_t cols, float* __restrict__ out, int64_t ldo, int accumulate);

// Host-side launcher.  a_kcontig / b_kcontig: the operand is contiguous along k.
mtgnn_status gemm_launch(const GemmArgs& g, int dtype_a, int dtype_b, bool a_kcontig, bool b_kcontig, int ksplit,
                         hipStream_t s);

// Convenience wrappers for the three linear-layer products (row-major matrices).
// y[M,N] (+)= x[M,K] W[N,K]^T + bias
// pre_relu: store the pre-activation there and relu(y) in y.  round_bf16: round y to bfloat16.
mtgnn_status linear_fwd(const void* x, int x_dtype, int64_t ldx, const void* W, int w_dtype, int64_t ldw,
                        const float* bias, float* y, int64_t ldy, int64_t M, const int32_t* M_dev, int64_t N,
                        int64_t K, bool accumulate, hipStream_t s, float* pre_relu = nullptr, int64_t ldpre = 0,
                        bool round_bf16 = false);
// dx[M,K] (+)= dy[M,N] W[N,K]; gate: dx *= (gate > 0) elementwise (after accumulation)
mtgnn_status linear_dx(const float* dy, int64_t lddy, const void* W, int w_dtype, int64_t ldw, float* dx,
                       int64_t lddx, int64_t M, const int32_t* M_dev, int64_t N, int64_t K, bool accumulate,
                       hipStream_t s, const float* gate = nullptr, int64_t ldgate = 0);
// dW[N,K] = dy[R,N]^T x[R,K], reduction over R rows (clamped by R_dev), split-K through ws.
size_t linear_dw_ws_bytes(int64_t R, int64_t N, int64_t K);
mtgnn_status linear_dw(const float* dy, int64_t lddy, const void* x, int x_dtype, int64_t ldx, float* dW,
                       int64_t lddw, int64_t R, const int32_t* R_dev, int64_t N, int64_t K, void* ws,
                       size_t ws_bytes, hipStream_t s);

}  // namespace mtgnn

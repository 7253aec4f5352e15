// Fused merge-layer chains of the attention embedding (float32).
//
// Forward, per query row (a = attention output, h = M[q], o stored in m_in[:, :da]):
//   o  = W_o a + b_o;   m1 = W_1 [o || h] + b_1;   a1 = relu(m1);   z = W_2 a1 + b_2
// Backward, from dz:
//   dm1 = (W_2^T dz) * [m1 > 0];   dm_in = W_1^T dm1;   dattn = W_o^T dm_in[:, :da]
//
// Each chain runs as one kernel instead of three products, every output the
// backward needs still written to memory.  A block of four waves owns a 16-row
// tile: the activations sit in LDS, shared by the waves, and each wave computes
// every fourth 16-column output tile of a layer, with a block barrier between
// layers.  A layer Y = X B^T (B row-major [N, K]: W for the forward, the
// transposed copies W^T for the backward) runs as 16-deep k chunks of
// v_mfma_f32_16x16x4_f32: lane l reads X[l%16][16 c + 4 (l/16) ..] from LDS and
// B[16 t + l%16][16 c + 4 (l/16) ..] from memory (the weights stay in L2),
// several chunks of weight fragments in flight ahead of the MFMAs.
#include <algorithm>
#include <type_traits>

#include "gemm.h"
#include "ops.h"

namespace mtgnn {

namespace {

constexpr int XS = 212;   // LDS row stride (floats) of an activation tile: >= 208, XS / 4 odd (conflict-free rows)
constexpr int MW = 4;     // waves per block; wave w computes the output column tiles w, w + 4, ...
constexpr int PD = 3;     // weight chunks in flight ahead of the one being multiplied (6 measured slower)

constexpr int RT1 = 1;   // row tiles per block of the single-layer kernels (query projection, d M', GRU dx);
                          // 2 (half the weight-fragment loads per row) measured slower: half the blocks

template <int NCT> struct Tiles { static constexpr int per_wave = (NCT + MW - 1) / MW; };

// acc[r NU + u] (16 x 16 output tile t = wave + 4 u of row tile r) += X[16 rows of tile r, 16 KC]
// B[16 t.., 16 KC]^T.  X: the block's LDS tile of 16 RT rows (row stride XSS, zero beyond the true width).
// B: a zero-padded weight copy, 16 MW NU rows by 16 KC columns, so every fragment load is in bounds and
// unconditional; each fragment serves the RT row tiles.
template <int NCT, int KC, int XSS = XS, int RT = 1>
__device__ __forceinline__ void layer(const float* X, const float* __restrict__ B,
                                      f32x4 (&acc)[RT * Tiles<NCT>::per_wave]) {
  constexpr int NU = Tiles<NCT>::per_wave;
  constexpr int LDB = 16 * KC;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, fr = lane & 15, fg = lane >> 4;
#pragma unroll
  for (int u = 0; u < RT * NU; ++u) acc[u] = f32x4{0.f, 0.f, 0.f, 0.f};
  const float* Bl = B + (16 * wid + fr) * LDB + 4 * fg;
  float4 bf[KC][NU];
  auto load_b = [&](int c) {
#pragma unroll
    for (int u = 0; u < NU; ++u) bf[c][u] = *reinterpret_cast<const float4*>(Bl + 16 * MW * u * LDB + 16 * c);
  };
#pragma unroll
  for (int c = 0; c < PD && c < KC; ++c) load_b(c);
#pragma unroll
  for (int c = 0; c < KC; ++c) {
    if (c + PD < KC) load_b(c + PD);   // in flight while this chunk's MFMAs run
#pragma unroll
    for (int r = 0; r < RT; ++r) {
      const float4 a = *reinterpret_cast<const float4*>(X + (16 * r + fr) * XSS + 16 * c + 4 * fg);
#pragma unroll
      for (int u = 0; u < NU; ++u) {
        f32x4& d = acc[r * NU + u];
        d = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, bf[c][u].x, d, 0, 0, 0);
        d = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, bf[c][u].y, d, 0, 0, 0);
        d = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, bf[c][u].z, d, 0, 0, 0);
        d = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, bf[c][u].w, d, 0, 0, 0);
      }
    }
    __builtin_amdgcn_sched_barrier(0);   // keeps the prefetch distance as written
  }
}

// rows r0 .. r0 + 16 RT - 1 (those < M) of a row-major [M, n] matrix into an LDS tile at column offset col0
template <int XSS = XS, int RT = 1>
__device__ __forceinline__ void load_rows(float* X, int col0, const float* __restrict__ src, int64_t ld, int n,
                                          int64_t r0, int64_t M) {
  const int nq = n / 4;
  for (int e = threadIdx.x; e < 16 * RT * nq; e += 64 * MW) {
    const int r = e / nq, q = e % nq;
    const float4 v = r0 + r < M ? *reinterpret_cast<const float4*>(src + (r0 + r) * ld + 4 * q)
                                : float4{0.f, 0.f, 0.f, 0.f};
    *reinterpret_cast<float4*>(X + r * XSS + col0 + 4 * q) = v;
  }
}

template <int XSS = XS, int RT = 1>
__device__ __forceinline__ void zero_cols(float* X, int c0, int c1) {
  for (int e = threadIdx.x; e < 16 * RT * (c1 - c0); e += 64 * MW)
    X[(e / (c1 - c0)) * XSS + c0 + e % (c1 - c0)] = 0.f;
}

// Epilogue of a layer: f(i, j, row valid, value) for this wave's tiles, row 16 t + 4 (l/16) + r of row tile
// t, column 16 u' + l%16 (j < N only).  A full block of rows takes a path with the row test folded away.
template <int NCT, int RT = 1, class F>
__device__ __forceinline__ void each_out(const f32x4 (&acc)[RT * Tiles<NCT>::per_wave], int N, int64_t r0,
                                         int64_t M, F f) {
  constexpr int NU = Tiles<NCT>::per_wave;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, fr = lane & 15, fg = lane >> 4;
  auto run = [&](auto full) {
#pragma unroll
    for (int t = 0; t < RT; ++t)
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      const int j = 16 * (wid + MW * u) + fr;
      if (j >= N) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = 16 * t + 4 * fg + r;
        f(i, j, decltype(full)::value || r0 + i < M, acc[t * NU + u][r]);
      }
    }
  };
  if (r0 + 16 * RT <= M)
    run(std::true_type{});
  else
    run(std::false_type{});
}

// NA = ceil(da / 16), NS = ceil((da + dm) / 16)
template <int NA, int NS>
__global__ __launch_bounds__(64 * MW) void k_merge_fwd(const float* __restrict__ attn, float* __restrict__ m_in,
                                                       const float* __restrict__ Wo, const float* __restrict__ bo,
                                                       const float* __restrict__ W1, const float* __restrict__ b1,
                                                       const float* __restrict__ W2, const float* __restrict__ b2,
                                                       float* __restrict__ m1, float* __restrict__ a1,
                                                       float* __restrict__ z, const int32_t* __restrict__ n_q,
                                                       int64_t max_q, int da, int dm) {
  __shared__ __attribute__((aligned(16))) float X0[16 * XS], X1[16 * XS];
  const int64_t M = eff_count(max_q, n_q);
  const int64_t r0 = (int64_t)blockIdx.x * 16;
  if (r0 >= M) return;   // block-uniform
  const int ldm = da + dm;
  zero_cols(X0, da, 16 * NS);
  zero_cols(X1, ldm, 16 * NS);
  load_rows(X0, 0, attn, da, da, r0, M);
  load_rows(X1, da, m_in + da, ldm, dm, r0, M);   // h = M[q], written by the query gather
  __syncthreads();
  f32x4 acc[Tiles<NA>::per_wave];
  // o = W_o a + b_o  -> m_in[:, :da] and X1[:, :da]
  layer<NA, NA>(X0, Wo, acc);
  each_out<NA>(acc, da, r0, M, [&](int i, int j, bool ok, float v) {
    v += bo[j];
    if (ok) m_in[(r0 + i) * ldm + j] = v;
    X1[i * XS + j] = v;
  });
  __syncthreads();
  // m1 = W_1 [o || h] + b_1;  a1 = relu(m1)  -> m1, a1 and X0[:, :da]  (X0 is no longer read)
  layer<NA, NS>(X1, W1, acc);
  each_out<NA>(acc, da, r0, M, [&](int i, int j, bool ok, float v) {
    v += b1[j];
    const float r = fmaxf(v, 0.f);
    if (ok) {
      m1[(r0 + i) * da + j] = v;
      a1[(r0 + i) * da + j] = r;
    }
    X0[i * XS + j] = r;
  });
  __syncthreads();
  // z = W_2 a1 + b_2
  layer<NA, NA>(X0, W2, acc);
  each_out<NA>(acc, da, r0, M, [&](int i, int j, bool ok, float v) {
    if (ok) z[(r0 + i) * da + j] = v + b2[j];
  });
}

// W2t = W_2^T [da, da], W1t = W_1^T [da + dm, da], Wot = W_o^T [da, da]
template <int NA, int NS>
__global__ __launch_bounds__(64 * MW) void k_merge_bwd(const float* __restrict__ dz, const float* __restrict__ W2t,
                                                       const float* __restrict__ W1t, const float* __restrict__ Wot,
                                                       const float* __restrict__ m1, float* __restrict__ dm1,
                                                       float* __restrict__ dm_in, float* __restrict__ dattn,
                                                       const int32_t* __restrict__ n_q, int64_t max_q, int da,
                                                       int dm) {
  __shared__ __attribute__((aligned(16))) float X0[16 * XS], X1[16 * XS];
  const int64_t M = eff_count(max_q, n_q);
  const int64_t r0 = (int64_t)blockIdx.x * 16;
  if (r0 >= M) return;   // block-uniform
  const int ldm = da + dm;
  zero_cols(X0, da, 16 * NS);
  zero_cols(X1, da, 16 * NS);
  load_rows(X0, 0, dz, da, da, r0, M);
  __syncthreads();
  // dm1 = (W_2^T dz) * [m1 > 0]  -> dm1 and X1[:, :da]
  {
    f32x4 acc[Tiles<NA>::per_wave];
    layer<NA, NA>(X0, W2t, acc);
    each_out<NA>(acc, da, r0, M, [&](int i, int j, bool ok, float v) {
      if (ok) {
        v = m1[(r0 + i) * da + j] > 0.f ? v : 0.f;
        dm1[(r0 + i) * da + j] = v;
      } else {
        v = 0.f;
      }
      X1[i * XS + j] = v;
    });
  }
  __syncthreads();
  // dm_in = W_1^T dm1  -> dm_in [.., da + dm] and X0[:, :da]  (X0 is no longer read)
  {
    f32x4 acc[Tiles<NS>::per_wave];
    layer<NS, NA>(X1, W1t, acc);
    each_out<NS>(acc, ldm, r0, M, [&](int i, int j, bool ok, float v) {
      if (ok) dm_in[(r0 + i) * ldm + j] = v;
      if (j < da) X0[i * XS + j] = v;
    });
  }
  __syncthreads();
  // dattn = W_o^T dm_in[:, :da]
  {
    f32x4 acc[Tiles<NA>::per_wave];
    layer<NA, NA>(X0, Wot, acc);
    each_out<NA>(acc, da, r0, M, [&](int i, int j, bool ok, float v) {
      if (ok) dattn[(r0 + i) * da + j] = v;
    });
  }
}

// Zero-padded copies of the merge weights: dst[r][c] = W[r][c] (or W[c][r] for a transposed copy) for r < n,
// c < k, else 0.  blockIdx.y selects the copy.
constexpr int PREP_MAX = 14;   // the six merge copies and up to eight extra copies
struct PrepArgs {
  const float* src[PREP_MAX];
  float* dst[PREP_MAX];
  int rows[PREP_MAX], cols[PREP_MAX], n[PREP_MAX], k[PREP_MAX], ld[PREP_MAX], tr[PREP_MAX], ldd[PREP_MAX];
  int ncopy;   // copies; grid slice ncopy (if present) forms the query constant
  QConst qc;
};

__global__ void k_merge_prepare(PrepArgs a) {
  const int m = blockIdx.y;
  if (m == a.ncopy) {   // the query constant c_j = b_q[j] + sum_t W_q[j][dm + t] phi(0)_t, a wave per j
    const QConst& q = a.qc;
    const int lane = threadIdx.x & 63;
    const int Dq = q.dm + q.dt;
    for (int j = blockIdx.x * 4 + (threadIdx.x >> 6); j < q.da; j += gridDim.x * 4) {
      float v = 0.f;
      for (int t = lane; t < q.dt; t += 64) v += q.Wq[(int64_t)j * Dq + q.dm + t] * cosf(time_arg(q.tw[t], 0.f, q.tb[t]));
      v = wave_sum(v);
      if (lane == 0) q.out[j] = q.bq[j] + v;
    }
    return;
  }
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= (int64_t)a.rows[m] * a.cols[m]) return;
  const int r = (int)(e / a.cols[m]), c = (int)(e % a.cols[m]);
  float v = 0.f;
  if (r < a.n[m] && c < a.k[m]) v = a.tr[m] ? a.src[m][(int64_t)c * a.ld[m] + r] : a.src[m][(int64_t)r * a.ld[m] + c];
  a.dst[m][(int64_t)r * a.ldd[m] + c] = v;
}

// Layout of the padded copies in one buffer: forward W_o, W_1, W_2, then backward W_2^T, W_1^T, W_o^T.
struct PackLayout {
  int rows[6], cols[6];
  size_t off[7];
  PackLayout(int da, int dm) {
    const int na = (int)cdiv(da, 16), ns = (int)cdiv(da + dm, 16);
    auto R = [](int nct) { return 16 * MW * (int)cdiv(nct, MW); };
    const int r[6] = {R(na), R(na), R(na), R(na), R(ns), R(na)};
    const int c[6] = {16 * na, 16 * ns, 16 * na, 16 * na, 16 * na, 16 * na};
    off[0] = 0;
    for (int m = 0; m < 6; ++m) {
      rows[m] = r[m];
      cols[m] = c[m];
      off[m + 1] = off[m] + (size_t)r[m] * c[m];
    }
  }
};

// The query projection's padded copies, after the merge copies: W_q[:, :d_m] (d_a rows, d_m columns:
// a query's time input is the constant phi(0), whose share is added as a bias) and W_q[:, :d_m]^T
// (d_m rows, d_a columns);
// and W_kv[:, :d_m]^T (d_m rows, 2 d_a columns: the d M' product over the summed dK|dV).
struct QLayout {
  int na, nm, kk;
  int rows[3], cols[3];
  size_t off[4];
  QLayout(int da, int dm, int dt) {
    na = (int)cdiv(da, 16);
    nm = (int)cdiv(dm, 16);
    kk = (int)cdiv(2 * da, 16);
    auto R = [](int nct) { return 16 * MW * (int)cdiv(nct, MW); };
    rows[0] = R(na);
    cols[0] = 16 * nm;
    rows[1] = R(nm);
    cols[1] = 16 * na;
    rows[2] = R(nm);
    cols[2] = 16 * kk;
    off[0] = PackLayout(da, dm).off[6];
    for (int m = 0; m < 3; ++m) off[m + 1] = off[m] + (size_t)rows[m] * cols[m];
  }
};

// qv = W_q [M[q] || phi(0)] + b_q over 16-row tiles of the queries.  The time input phi(0) = cos(b) is
// the same for every query, so qv = W_q[:, :dm] M[q] + c with c = b_q + W_q[:, dm:] phi(0) (formed
// once by the weight preparation): the product runs over the dm memory columns of q_in (row stride
// D_q).  Wp: W_q[:, :dm] padded.
template <int NA, int KM>
__global__ __launch_bounds__(64 * MW) void k_qproj_fwd(const float* __restrict__ q_in, const float* __restrict__ Wp,
                                                       const float* __restrict__ cq, float* __restrict__ qv,
                                                       const int32_t* __restrict__ n_q, int64_t max_q, int da, int dm,
                                                       int Dq) {
  __shared__ __attribute__((aligned(16))) float X0[16 * RT1 * XS];
  const int64_t M = eff_count(max_q, n_q);
  const int64_t r0 = (int64_t)blockIdx.x * 16 * RT1;
  if (r0 >= M) return;   // block-uniform
  zero_cols<XS, RT1>(X0, dm, 16 * KM);
  load_rows<XS, RT1>(X0, 0, q_in, Dq, dm, r0, M);
  __syncthreads();
  f32x4 acc[RT1 * Tiles<NA>::per_wave];
  layer<NA, KM, XS, RT1>(X0, Wp, acc);
  each_out<NA, RT1>(acc, da, r0, M, [&](int i, int j, bool ok, float v) {
    if (ok) qv[(r0 + i) * da + j] = v + cq[j];
  });
}

// dm_in[:, da:] += dqv W_q[:, :dm] (the memory part of the query input), WqT = W_q[:, :dm]^T padded.
template <int NM, int NA>
__global__ __launch_bounds__(64 * MW) void k_qproj_dx(const float* __restrict__ dqv, const float* __restrict__ WqT,
                                                      float* __restrict__ dm_in, int64_t ldm,
                                                      const int32_t* __restrict__ n_q, int64_t max_q, int da, int dm) {
  __shared__ __attribute__((aligned(16))) float X0[16 * RT1 * XS];
  const int64_t M = eff_count(max_q, n_q);
  const int64_t r0 = (int64_t)blockIdx.x * 16 * RT1;
  if (r0 >= M) return;   // block-uniform
  zero_cols<XS, RT1>(X0, da, 16 * NA);
  load_rows<XS, RT1>(X0, 0, dqv, da, da, r0, M);
  __syncthreads();
  f32x4 acc[RT1 * Tiles<NM>::per_wave];
  layer<NM, NA, XS, RT1>(X0, WqT, acc);
  each_out<NM, RT1>(acc, dm, r0, M, [&](int i, int j, bool ok, float v) {
    if (ok) dm_in[(r0 + i) * ldm + da + j] += v;
  });
}

// d_mem[:, :dm] += S[:, dm : dm + 2 da] W_kv[:, :dm] over 16-row tiles (S: the per-row sums of
// [dh_q | dK | dV], row stride ldS; WkT = W_kv[:, :dm]^T padded).
template <int NM, int KK>
__global__ __launch_bounds__(64 * MW) void k_dmem_dx(const float* __restrict__ S, int64_t ldS,
                                                     const float* __restrict__ WkT, float* __restrict__ d_mem,
                                                     const int32_t* __restrict__ n_rows, int64_t max_rows, int dm,
                                                     int w2) {
  __shared__ __attribute__((aligned(16))) float X0[16 * RT1 * XS];
  const int64_t M = eff_count(max_rows, n_rows);
  const int64_t r0 = (int64_t)blockIdx.x * 16 * RT1;
  if (r0 >= M) return;   // block-uniform
  zero_cols<XS, RT1>(X0, w2, 16 * KK);
  load_rows<XS, RT1>(X0, 0, S + dm, ldS, w2, r0, M);
  __syncthreads();
  f32x4 acc[RT1 * Tiles<NM>::per_wave];
  layer<NM, KK, XS, RT1>(X0, WkT, acc);
  each_out<NM, RT1>(acc, dm, r0, M, [&](int i, int j, bool ok, float v) {
    if (ok) d_mem[(r0 + i) * dm + j] += v;
  });
}

// The GRU backward's time-feature gradient: dmsg_time = dgi W_ih[:, c0 : c0 + dt] over 16-row tiles of dgi
// (3 dm wide); WT = W_ih[:, c0 : c0 + dt]^T zero-padded (gru_dx_weight_copy).
constexpr int XS_GRU = 308;   // >= 304 (19 chunks of 16), XS_GRU / 4 odd

template <int NT, int KC>
__global__ __launch_bounds__(64 * MW) void k_gru_dx(const float* __restrict__ dgi, int64_t ldg,
                                                    const float* __restrict__ WT, float* __restrict__ out, int dt,
                                                    const int32_t* __restrict__ n_rows, int64_t max_rows, int K) {
  __shared__ __attribute__((aligned(16))) float X0[16 * RT1 * XS_GRU];
  const int64_t M = eff_count(max_rows, n_rows);
  const int64_t r0 = (int64_t)blockIdx.x * 16 * RT1;
  if (r0 >= M) return;   // block-uniform
  zero_cols<XS_GRU, RT1>(X0, K, 16 * KC);
  load_rows<XS_GRU, RT1>(X0, 0, dgi, ldg, K, r0, M);
  __syncthreads();
  f32x4 acc[RT1 * Tiles<NT>::per_wave];
  layer<NT, KC, XS_GRU, RT1>(X0, WT, acc);
  each_out<NT, RT1>(acc, dt, r0, M, [&](int i, int j, bool ok, float v) {
    if (ok) out[(r0 + i) * dt + j] = v;
  });
}

// ---------------------------------------------------------------- the GRU update on the layer machinery

// A block owns 16 updated rows and GRU_UNITS hidden units: the r, z and n columns of both products for
// those units (6 x 32 = 192 output columns; the padded weight copy of group g holds the r, z, n rows of
// its units, then 32 zero rows).  The message rows go to LDS once: the input product reads all of them,
// the hidden product their first d_mem columns (h = M[node], the message's first slice; the padded W_hh
// is zero past d_mem).  The six pre-activations meet in LDS and the gates are applied there.
constexpr int GRU_UNITS = 32;
constexpr int GRU_GROUP_ROWS = 128;   // 6 column tiles of the layer read 8 tiles' rows (16 MW NU)

// The padded per-group weights (float32): Wi [groups][128][16 ki], Wh [groups][128][16 kh]; row 32 gate + u
// of group g is unit 32 g + u of gate (r, z, n) = (0, 1, 2); rows 96..127, units past d_mem and columns past
// the true width are zero.  Side job: the backward's padded W_ih time slice (as the unfused gate kernel).
__global__ void k_gru_prepare(const float* __restrict__ W_ih, const float* __restrict__ W_hh, int dm, int dmsg,
                              int ki16, int kh16, int groups, float* __restrict__ Wi, float* __restrict__ Wh,
                              GruWTArgs wt) {
  const int64_t e0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x, stride = (int64_t)gridDim.x * blockDim.x;
  const int64_t ni = (int64_t)groups * GRU_GROUP_ROWS * ki16, nh = (int64_t)groups * GRU_GROUP_ROWS * kh16;
  for (int64_t x = e0; x < ni + nh; x += stride) {
    const bool in = x < ni;
    const int64_t y = in ? x : x - ni;
    const int kk = in ? ki16 : kh16;
    const int g = (int)(y / (GRU_GROUP_ROWS * kk));
    const int row = (int)(y / kk % GRU_GROUP_ROWS), col = (int)(y % kk);
    const int gate = row / GRU_UNITS, unit = GRU_UNITS * g + row % GRU_UNITS;
    const int K = in ? dmsg : dm;
    float v = 0.f;
    if (gate < 3 && unit < dm && col < K) v = (in ? W_ih : W_hh)[(int64_t)(gate * dm + unit) * K + col];
    (in ? Wi : Wh)[y] = v;
  }
  if (wt.dst)
    for (int64_t x = e0; x < (int64_t)wt.rows * wt.cols; x += stride) {
      const int rr = (int)(x / wt.cols), cc = (int)(x % wt.cols);
      wt.dst[x] = (rr < wt.dt && cc < wt.K) ? W_ih[(int64_t)cc * wt.ld + wt.col0 + rr] : 0.f;
    }
}

template <int KI, int KH>
__global__ __launch_bounds__(64 * MW) void k_gru_fused(const float* __restrict__ msg, int dmsg,
                                                       const float* __restrict__ Wi, const float* __restrict__ Wh,
                                                       const float* __restrict__ b_ih, const float* __restrict__ b_hh,
                                                       const int32_t* __restrict__ uniq,
                                                       const int32_t* __restrict__ winner, const float* __restrict__ t,
                                                       const int32_t* __restrict__ n_rows, int64_t max_rows, int dm,
                                                       float* __restrict__ mem, float* __restrict__ lu,
                                                       float* __restrict__ sr, float* __restrict__ sz,
                                                       float* __restrict__ sn, float* __restrict__ sghn) {
  constexpr int XL = 16 * KI + 4;   // LDS row stride, XL / 4 odd
  constexpr int GL = 6 * GRU_UNITS + 4;
  __shared__ __attribute__((aligned(16))) float X[16 * XL];
  __shared__ float G[16 * GL];
  const int64_t M = eff_count(max_rows, n_rows);
  const int64_t r0 = (int64_t)blockIdx.x * 16;
  if (r0 >= M) return;   // block-uniform
  const int g = blockIdx.y;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, fr = lane & 15, fg = lane >> 4;
  zero_cols<XL, 1>(X, dmsg, 16 * KI);
  load_rows<XL, 1>(X, 0, msg, dmsg, dmsg, r0, M);
  __syncthreads();
  {
    f32x4 ai[Tiles<6>::per_wave], ah[Tiles<6>::per_wave];
    layer<6, KI, XL, 1>(X, Wi + (size_t)g * GRU_GROUP_ROWS * 16 * KI, ai);
    layer<6, KH, XL, 1>(X, Wh + (size_t)g * GRU_GROUP_ROWS * 16 * KH, ah);
#pragma unroll
    for (int u = 0; u < Tiles<6>::per_wave; ++u) {
      const int c = 16 * (wid + MW * u) + fr;
      if (c >= 3 * GRU_UNITS) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        G[(4 * fg + r) * GL + c] = ai[u][r];
        G[(4 * fg + r) * GL + 3 * GRU_UNITS + c] = ah[u][r];
      }
    }
  }
  __syncthreads();
  for (int e = threadIdx.x; e < 16 * GRU_UNITS; e += 64 * MW) {
    const int i = e / GRU_UNITS, jj = e % GRU_UNITS, j = GRU_UNITS * g + jj;
    if (j >= dm || r0 + i >= M) continue;
    const float* gi = G + i * GL;
    const float* gh = gi + 3 * GRU_UNITS;
    const float rr = sigmoidf_((gi[jj] + b_ih[j]) + (gh[jj] + b_hh[j]));
    const float zz = sigmoidf_((gi[GRU_UNITS + jj] + b_ih[dm + j]) + (gh[GRU_UNITS + jj] + b_hh[dm + j]));
    const float ghn = gh[2 * GRU_UNITS + jj] + b_hh[2 * dm + j];
    const float nn = tanhf((gi[2 * GRU_UNITS + jj] + b_ih[2 * dm + j]) + rr * ghn);
    const float h = X[i * XL + j];
    const float hn = (1.f - zz) * nn + zz * h;
    const int64_t row = r0 + i;
    const int64_t node = uniq[row];
    mem[node * dm + j] = hn;
    if (j == 0) lu[node] = t[winner[row] >> 1];
    if (sr) {
      sr[row * dm + j] = rr;
      sz[row * dm + j] = zz;
      sn[row * dm + j] = nn;
      sghn[row * dm + j] = ghn;
    }
  }
}

// ---------------------------------------------------------------- the link-prediction decoder

// One block per 16 target events (their src, dst and negative query rows of z).  Forward:
//   pre_pos = W_a z_src + W_b z_dst + b_d1,  pre_neg = W_a z_src + W_b z_neg + b_d1,
//   s = W_d2 relu(pre) + b_d2,  l = softplus(-s_pos) + softplus(s_neg);
// backward: ds_pos = (sigmoid(s_pos) - 1) / n, ds_neg = sigmoid(s_neg) / n, dh = ds W_d2 [pre > 0],
//   dz_src = (dh_pos + dh_neg) W_a, dz_dst = dh_pos W_b, dz_neg = dh_neg W_b.
// W_a, W_b are the column halves of W_d1; Wp holds their zero-padded copies and transposes.  The
// hidden-row gradients also go to the query-layout buffers DA (src rows: dh_pos + dh_neg, other rows
// zero) and DB (dst rows dh_pos, neg rows dh_neg, src rows zero), for dW_d1 = [DA^T z | DB^T z];
// part[block] = the block's sums of ds_pos h_pos + ds_neg h_neg (d_a), ds_pos + ds_neg, and l / n.
template <int NA>
__global__ __launch_bounds__(64 * MW) void k_link_fused(const float* __restrict__ z, const int32_t* __restrict__ n_q,
                                                        int64_t max_tar, int da, const float* __restrict__ Wp,
                                                        const float* __restrict__ b1, const float* __restrict__ W2,
                                                        const float* __restrict__ b2, float* __restrict__ DA,
                                                        float* __restrict__ DB, float* __restrict__ dz,
                                                        float* __restrict__ scores, float* __restrict__ part) {
  constexpr int XL = 16 * NA + 4;   // LDS row stride: >= 16 NA, XL / 4 odd
  constexpr int NU = Tiles<NA>::per_wave;
  constexpr size_t WSZ = (size_t)16 * MW * NU * 16 * NA;   // floats per padded copy
  __shared__ __attribute__((aligned(16))) float T[5][16 * XL];   // z_src, z_dst, z_neg (then dh), pre_pos, pre_neg
  __shared__ float red[MW][2 * 64 + 2];
  const int64_t n = (n_q ? (int64_t)*n_q : 3 * max_tar) / 3;
  const int64_t r0 = (int64_t)blockIdx.x * 16;
  if (r0 >= n) return;   // block-uniform
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, fr = lane & 15, fg = lane >> 4;
  for (int b = 0; b < 3; ++b) {
    zero_cols<XL, 1>(T[b], da, 16 * NA);
    load_rows<XL, 1>(T[b], 0, z + (int64_t)b * n * da, da, da, r0, n);
  }
  __syncthreads();
  {
    f32x4 as[NU], ad[NU], an[NU];
    layer<NA, NA, XL, 1>(T[0], Wp, as);
    layer<NA, NA, XL, 1>(T[1], Wp + WSZ, ad);
    layer<NA, NA, XL, 1>(T[2], Wp + WSZ, an);
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      const int j = 16 * (wid + MW * u) + fr;
      if (j >= 16 * NA) continue;
      const float bj = j < da ? b1[j] : 0.f;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = 4 * fg + r;
        T[3][i * XL + j] = (as[u][r] + ad[u][r]) + bj;
        T[4][i * XL + j] = (as[u][r] + an[u][r]) + bj;
      }
    }
  }
  __syncthreads();
  // scores, loss terms and hidden-row gradients: wave w takes events 4w .. 4w + 3
  const float inv_n = 1.0f / (float)n;
  float gsum[2] = {0.f, 0.f}, dsum = 0.f, lsum = 0.f;
  float w2[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) w2[h] = lane + 64 * h < da ? W2[lane + 64 * h] : 0.f;
  for (int e = 4 * wid; e < 4 * wid + 4; ++e) {
    const bool ok = r0 + e < n;
    float sp = 0.f, sn = 0.f;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int j = lane + 64 * h;
      if (j < da) {
        sp += w2[h] * fmaxf(T[3][e * XL + j], 0.f);
        sn += w2[h] * fmaxf(T[4][e * XL + j], 0.f);
      }
    }
    sp = wave_sum(sp) + b2[0];
    sn = wave_sum(sn) + b2[0];
    const float dsp = ok ? (1.0f / (1.0f + expf(-sp)) - 1.0f) * inv_n : 0.f;
    const float dsn = ok ? (1.0f / (1.0f + expf(-sn))) * inv_n : 0.f;
    const int64_t q = r0 + e;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int j = lane + 64 * h;
      if (j < 16 * NA) {
        const float pp = T[3][e * XL + j], pn = T[4][e * XL + j];
        const float dhp = (j < da && pp > 0.f) ? dsp * w2[h] : 0.f;
        const float dhn = (j < da && pn > 0.f) ? dsn * w2[h] : 0.f;
        T[0][e * XL + j] = dhp + dhn;
        T[1][e * XL + j] = dhp;
        T[2][e * XL + j] = dhn;
        if (ok && j < da) {
          DA[q * da + j] = dhp + dhn;
          DA[(n + q) * da + j] = 0.f;
          DA[(2 * n + q) * da + j] = 0.f;
          DB[q * da + j] = 0.f;
          DB[(n + q) * da + j] = dhp;
          DB[(2 * n + q) * da + j] = dhn;
          gsum[h] += dsp * fmaxf(pp, 0.f) + dsn * fmaxf(pn, 0.f);
        }
      }
    }
    if (ok) {
      dsum += dsp + dsn;
      lsum += (fmaxf(-sp, 0.f) + log1pf(expf(-fabsf(sp)))) * inv_n + (fmaxf(sn, 0.f) + log1pf(expf(-fabsf(sn)))) * inv_n;
      if (scores && lane == 0) {
        scores[q] = sp;
        scores[max_tar + q] = sn;
      }
    }
  }
  red[wid][lane] = gsum[0];
  red[wid][64 + lane] = gsum[1];
  if (lane == 0) {
    red[wid][128] = dsum;
    red[wid][129] = lsum;
  }
  __syncthreads();
  // the block's partial sums, the four waves added in a fixed order
  for (int c = threadIdx.x; c < da + 2; c += 64 * MW) {
    const int k = c < da ? c : 128 + (c - da);
    part[(int64_t)blockIdx.x * (da + 2) + c] = ((red[0][k] + red[1][k]) + red[2][k]) + red[3][k];
  }
  // dz for the three query blocks
  for (int b = 0; b < 3; ++b) {
    f32x4 acc[NU];
    layer<NA, NA, XL, 1>(T[b], Wp + (b == 0 ? 2 : 3) * WSZ, acc);
    float* out = dz + (int64_t)b * n * da;
    each_out<NA, 1>(acc, da, r0, n, [&](int i, int j, bool ok, float v) {
      if (ok) out[(r0 + i) * da + j] = v;
    });
  }
}

// Column sums of the partials of the blocks that hold target events (cdiv(n_tar, 16)), in a fixed order,
// a wave per column: dW_d2, db_d2 and the loss.
__global__ __launch_bounds__(256) void k_link_reduce_dev(const float* __restrict__ part,
                                                         const int32_t* __restrict__ n_q, int64_t max_tar, int da,
                                                         float* __restrict__ dW2, float* __restrict__ db2,
                                                         float* __restrict__ loss) {
  const int c = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (c >= da + 2) return;
  const int64_t n = (n_q ? (int64_t)*n_q : 3 * max_tar) / 3;
  const int64_t nblk = cdiv(n, 16);
  float v = 0.f;
  for (int64_t b = lane; b < nblk; b += 64) v += part[b * (da + 2) + c];
  v = wave_sum(v);
  if (lane == 0) {
    if (c < da) dW2[c] = v;
    else if (c == da) db2[0] = v;
    else loss[0] = v;
  }
}

bool aligned16(const void* p) { return ((uintptr_t)p % 16) == 0; }

}  // namespace

// Shapes of the fused GRU time-feature gradient: 3 dm in (288, 304] or (80, 96], dt tiles 7 or 2.
bool gru_dx_fused_ok(int dtype, int dm, int dt) {
  const int kc = (int)cdiv(3 * dm, 16), nt = (int)cdiv(dt, 16);
  return dtype == MTGNN_F32 && dm % 4 == 0 && dt % 4 == 0 && ((kc == 19 && nt == 7) || (kc == 6 && nt == 2));
}

size_t gru_dx_weight_floats(int dm, int dt) {
  return (size_t)16 * MW * cdiv(cdiv(dt, 16), MW) * 16 * cdiv(3 * dm, 16);
}

mtgnn_status gru_dx_fused(const float* dgi, const float* WT, float* dmsg_time, const int32_t* n_rows,
                          int64_t max_rows, int dm, int dt, hipStream_t s) {
  if (max_rows <= 0) return MTGNN_OK;
  if (!aligned16(dgi) || !aligned16(WT)) return MTGNN_EUNSUPPORTED;
  const unsigned grid = (unsigned)cdiv(max_rows, 16 * RT1);
  if (cdiv(3 * dm, 16) == 19)
    k_gru_dx<7, 19><<<grid, 64 * MW, 0, s>>>(dgi, 3 * dm, WT, dmsg_time, dt, n_rows, max_rows, 3 * dm);
  else
    k_gru_dx<2, 6><<<grid, 64 * MW, 0, s>>>(dgi, 3 * dm, WT, dmsg_time, dt, n_rows, max_rows, 3 * dm);
  MTGNN_CHECK_LAUNCH("gru_dx");
  return MTGNN_OK;
}

bool qproj_fused_ok(int dtype, int da, int dm, int dt) {
  if (!merge_fused_ok(dtype, da, dm) || dt % 4 != 0) return false;
  const QLayout L(da, dm, dt);
  return (L.na == 7 && L.nm == 7 && L.kk == 13) || (L.na == 2 && L.nm == 2 && L.kk == 4);
}

bool merge_fused_ok(int dtype, int da, int dm) {
  const int na = (int)cdiv(da, 16), ns = (int)cdiv(da + dm, 16);
  return dtype == MTGNN_F32 && da % 4 == 0 && dm % 4 == 0 && ((na == 7 && ns == 13) || (na == 2 && ns == 4));
}

size_t merge_weights_floats(int da, int dm, int dt) {
  return qproj_fused_ok(MTGNN_F32, da, dm, dt) ? QLayout(da, dm, dt).off[3] : PackLayout(da, dm).off[6];
}

PadCopy qproj_copy(const float* Wq, int da, int dm, int dt, float* Wp, int which) {
  const QLayout L(da, dm, dt);
  if (which == 0) return PadCopy{Wq, Wp + L.off[0], L.rows[0], L.cols[0], da, dm, dm + dt, 0, 0};
  return PadCopy{Wq, Wp + L.off[1], L.rows[1], L.cols[1], dm, da, dm + dt, 1, 0};
}

PadCopy dmem_copy(const float* Wk, const float* Wv, int da, int dm, int dt, int Dkv, float* Wp, int which) {
  // the d M' product's W_kv[:, :dm]^T: its first d_a columns from W_k, the rest from W_v (and zeros)
  const QLayout L(da, dm, dt);
  float* base = Wp + L.off[2];
  if (which == 0) return PadCopy{Wk, base, L.rows[2], da, dm, da, Dkv, 1, L.cols[2]};
  return PadCopy{Wv, base + da, L.rows[2], L.cols[2] - da, dm, da, Dkv, 1, L.cols[2]};
}

mtgnn_status dmem_dx_fused(const float* S, int64_t ldS, const float* Wp, float* d_mem, const int32_t* n_rows,
                           int64_t max_rows, int da, int dm, int dt, hipStream_t s) {
  if (max_rows <= 0) return MTGNN_OK;
  if (!aligned16(S) || !aligned16(Wp) || (dm * sizeof(float)) % 16 != 0 || ldS % 4 != 0) return MTGNN_EUNSUPPORTED;
  const QLayout L(da, dm, dt);
  const unsigned grid = (unsigned)cdiv(max_rows, 16 * RT1);
  if (L.nm == 7)
    k_dmem_dx<7, 13><<<grid, 64 * MW, 0, s>>>(S, ldS, Wp + L.off[2], d_mem, n_rows, max_rows, dm, 2 * da);
  else
    k_dmem_dx<2, 4><<<grid, 64 * MW, 0, s>>>(S, ldS, Wp + L.off[2], d_mem, n_rows, max_rows, dm, 2 * da);
  MTGNN_CHECK_LAUNCH("dmem_dx");
  return MTGNN_OK;
}

mtgnn_status qproj_fwd_fused(const float* q_in, const float* Wp, const float* cq, float* qv, const int32_t* n_q,
                             int64_t max_q, int da, int dm, int dt, hipStream_t s) {
  if (max_q <= 0) return MTGNN_OK;
  if (!aligned16(q_in) || !aligned16(Wp) || (dm + dt) % 4 != 0) return MTGNN_EUNSUPPORTED;
  const QLayout L(da, dm, dt);
  const unsigned grid = (unsigned)cdiv(max_q, 16 * RT1);
  if (L.na == 7)
    k_qproj_fwd<7, 7><<<grid, 64 * MW, 0, s>>>(q_in, Wp + L.off[0], cq, qv, n_q, max_q, da, dm, dm + dt);
  else
    k_qproj_fwd<2, 2><<<grid, 64 * MW, 0, s>>>(q_in, Wp + L.off[0], cq, qv, n_q, max_q, da, dm, dm + dt);
  MTGNN_CHECK_LAUNCH("qproj_fwd");
  return MTGNN_OK;
}

mtgnn_status qproj_dx_fused(const float* dqv, const float* Wp, float* dm_in, int64_t ldm, const int32_t* n_q,
                            int64_t max_q, int da, int dm, int dt, hipStream_t s) {
  if (max_q <= 0) return MTGNN_OK;
  if (!aligned16(dqv) || !aligned16(Wp)) return MTGNN_EUNSUPPORTED;
  const QLayout L(da, dm, dt);
  const unsigned grid = (unsigned)cdiv(max_q, 16 * RT1);
  if (L.na == 7)
    k_qproj_dx<7, 7><<<grid, 64 * MW, 0, s>>>(dqv, Wp + L.off[1], dm_in, ldm, n_q, max_q, da, dm);
  else
    k_qproj_dx<2, 2><<<grid, 64 * MW, 0, s>>>(dqv, Wp + L.off[1], dm_in, ldm, n_q, max_q, da, dm);
  MTGNN_CHECK_LAUNCH("qproj_dx");
  return MTGNN_OK;
}

static bool gru_fused_shape(int dm, int dmsg, int& ki, int& kh) {
  ki = (int)cdiv(dmsg, 16);
  kh = (int)cdiv(dm, 16);
  return dm % 4 == 0 && dmsg % 4 == 0 &&
         ((ki == 19 && kh == 7) || (ki == 20 && kh == 7) || (ki == 30 && kh == 7) || (ki == 7 && kh == 2));
}

bool gru_fused_ok(int dtype, int dm, int dmsg) {
  int ki, kh;
  return dtype == MTGNN_F32 && gru_fused_shape(dm, dmsg, ki, kh);
}

size_t gru_fused_weight_floats(int dm, int dmsg) {
  const int64_t groups = cdiv(dm, GRU_UNITS);
  return (size_t)groups * GRU_GROUP_ROWS * 16 * (cdiv(dmsg, 16) + cdiv(dm, 16));
}

mtgnn_status gru_fused(const float* msg, const float* W_ih, const float* W_hh, const float* b_ih, const float* b_hh,
                       const int32_t* uniq, const int32_t* winner, const float* t, const int32_t* n_rows,
                       int64_t max_rows, int dm, int dmsg, float* Wp, float* mem, float* lu, float* sr, float* sz,
                       float* sn, float* sghn, GruWTArgs wt, hipStream_t s) {
  int ki, kh;
  if (!gru_fused_shape(dm, dmsg, ki, kh) || !aligned16(msg)) return MTGNN_EUNSUPPORTED;
  const int groups = (int)cdiv(dm, GRU_UNITS);
  float* Wi = Wp;
  float* Wh = Wp + (size_t)groups * GRU_GROUP_ROWS * 16 * ki;
  const int64_t tot = (int64_t)groups * GRU_GROUP_ROWS * 16 * (ki + kh);
  k_gru_prepare<<<(unsigned)std::min<int64_t>(cdiv(tot, 256), 1024), 256, 0, s>>>(W_ih, W_hh, dm, dmsg, 16 * ki,
                                                                                   16 * kh, groups, Wi, Wh, wt);
  MTGNN_CHECK_LAUNCH("gru_prepare");
  if (max_rows <= 0) return MTGNN_OK;
  const dim3 grid((unsigned)cdiv(max_rows, 16), (unsigned)groups);
#define MTGNN_GRU_FUSED(KI_, KH_)                                                                          \
  k_gru_fused<KI_, KH_><<<grid, 64 * MW, 0, s>>>(msg, dmsg, Wi, Wh, b_ih, b_hh, uniq, winner, t, n_rows, \
                                                  max_rows, dm, mem, lu, sr, sz, sn, sghn)
  if (ki == 19) MTGNN_GRU_FUSED(19, 7);
  else if (ki == 20) MTGNN_GRU_FUSED(20, 7);
  else if (ki == 30) MTGNN_GRU_FUSED(30, 7);
  else MTGNN_GRU_FUSED(7, 2);
#undef MTGNN_GRU_FUSED
  MTGNN_CHECK_LAUNCH("gru_fused");
  return MTGNN_OK;
}

bool link_fused_ok(int da) {
  const int na = (int)cdiv(da, 16);
  return da % 4 == 0 && (na == 7 || na == 2);
}

size_t link_fused_weight_floats(int da) {
  const int na = (int)cdiv(da, 16);
  return (size_t)4 * 16 * MW * cdiv(na, MW) * 16 * na;
}

mtgnn_status link_fused(const float* z, const int32_t* n_q, int64_t max_q, int da, const float* W1, const float* b1,
                        const float* W2, const float* b2, float* Wp, float* DA, float* DB, float* part, float* dz,
                        float* scores, float* dW2, float* db2, float* loss, hipStream_t s) {
  if (!link_fused_ok(da) || !aligned16(z) || !aligned16(Wp) || !aligned16(dz)) return MTGNN_EUNSUPPORTED;
  const int na = (int)cdiv(da, 16);
  const int rows = 16 * MW * (int)cdiv(na, MW), cols = 16 * na;
  const size_t wsz = (size_t)rows * cols;
  // zero-padded W_a, W_b (the column halves of W_d1) and their transposes
  PrepArgs a;
  for (int m = 0; m < 4; ++m) {
    a.src[m] = W1 + (m % 2 ? da : 0);
    a.dst[m] = Wp + m * wsz;
    a.rows[m] = rows;
    a.cols[m] = cols;
    a.n[m] = da;
    a.k[m] = da;
    a.ld[m] = 2 * da;
    a.tr[m] = m >= 2 ? 1 : 0;
    a.ldd[m] = cols;
  }
  a.ncopy = 4;
  k_merge_prepare<<<dim3((unsigned)cdiv(wsz, 256), 4u), 256, 0, s>>>(a);
  MTGNN_CHECK_LAUNCH("link_prepare");
  const int64_t max_tar = max_q / 3;
  const int64_t nblk = cdiv(max_tar < 1 ? 1 : max_tar, 16);
  if (max_tar > 0) {
    TimedScope ts("link_fused", s);
    if (na == 7)
      k_link_fused<7><<<(unsigned)nblk, 64 * MW, 0, s>>>(z, n_q, max_tar, da, Wp, b1, W2, b2, DA, DB, dz, scores,
                                                          part);
    else
      k_link_fused<2><<<(unsigned)nblk, 64 * MW, 0, s>>>(z, n_q, max_tar, da, Wp, b1, W2, b2, DA, DB, dz, scores,
                                                          part);
    MTGNN_CHECK_LAUNCH("link_fused");
  }
  // blocks past the device's target count wrote no partial: sum only those below it
  k_link_reduce_dev<<<(unsigned)cdiv(da + 2, 4), 256, 0, s>>>(part, n_q, max_tar, da, dW2, db2, loss);
  MTGNN_CHECK_LAUNCH("link_reduce");
  return MTGNN_OK;
}

mtgnn_status merge_prepare(const float* Wo, const float* W1, const float* W2, int da, int dm, float* Wp,
                           hipStream_t s, const PadCopy* extra, int n_extra, const QConst* qc) {
  if (n_extra < 0 || n_extra > PREP_MAX - 6) return MTGNN_EINVAL;
  const PackLayout L(da, dm);
  const int ldm = da + dm;
  PrepArgs a;
  const float* src[6] = {Wo, W1, W2, W2, W1, Wo};
  const int n[6] = {da, da, da, da, ldm, da}, k[6] = {da, ldm, da, da, da, da};
  const int ld[6] = {da, ldm, da, da, ldm, da}, tr[6] = {0, 0, 0, 1, 1, 1};
  int64_t most = 0;
  for (int m = 0; m < 6; ++m) {
    a.src[m] = src[m];
    a.dst[m] = Wp + L.off[m];
    a.rows[m] = L.rows[m];
    a.cols[m] = L.cols[m];
    a.n[m] = n[m];
    a.k[m] = k[m];
    a.ld[m] = ld[m];
    a.tr[m] = tr[m];
    a.ldd[m] = L.cols[m];
    most = std::max<int64_t>(most, (int64_t)L.rows[m] * L.cols[m]);
  }
  for (int x = 0; x < n_extra; ++x) {
    const int m = 6 + x;
    a.src[m] = extra[x].src;
    a.dst[m] = extra[x].dst;
    a.rows[m] = extra[x].rows;
    a.cols[m] = extra[x].cols;
    a.n[m] = extra[x].n;
    a.k[m] = extra[x].k;
    a.ld[m] = extra[x].ld;
    a.tr[m] = extra[x].tr;
    a.ldd[m] = extra[x].ldd > 0 ? extra[x].ldd : extra[x].cols;
    most = std::max<int64_t>(most, (int64_t)extra[x].rows * extra[x].cols);
  }
  a.ncopy = 6 + n_extra;
  if (qc) a.qc = *qc;
  k_merge_prepare<<<dim3((unsigned)cdiv(most, 256), (unsigned)(6 + n_extra + (qc ? 1 : 0))), 256, 0, s>>>(a);
  MTGNN_CHECK_LAUNCH("merge_prepare");
  return MTGNN_OK;
}

mtgnn_status merge_fwd_fused(const float* attn, float* m_in, const float* Wp, const float* bo, const float* b1,
                             const float* b2, float* m1, float* a1, float* z, const int32_t* n_q, int64_t max_q,
                             int da, int dm, hipStream_t s) {
  if (max_q <= 0) return MTGNN_OK;
  if (!aligned16(attn) || !aligned16(m_in) || !aligned16(Wp)) return MTGNN_EUNSUPPORTED;
  const PackLayout L(da, dm);
  const unsigned grid = (unsigned)cdiv(max_q, 16);
  TimedScope ts("merge_fwd", s);
  if (cdiv(da, 16) == 7)
    k_merge_fwd<7, 13><<<grid, 64 * MW, 0, s>>>(attn, m_in, Wp + L.off[0], bo, Wp + L.off[1], b1, Wp + L.off[2], b2,
                                                m1, a1, z, n_q, max_q, da, dm);
  else
    k_merge_fwd<2, 4><<<grid, 64 * MW, 0, s>>>(attn, m_in, Wp + L.off[0], bo, Wp + L.off[1], b1, Wp + L.off[2], b2,
                                               m1, a1, z, n_q, max_q, da, dm);
  MTGNN_CHECK_LAUNCH("merge_fwd");
  return MTGNN_OK;
}

mtgnn_status merge_bwd_fused(const float* dz, const float* Wp, const float* m1, float* dm1, float* dm_in,
                             float* dattn, const int32_t* n_q, int64_t max_q, int da, int dm, hipStream_t s) {
  if (max_q <= 0) return MTGNN_OK;
  if (!aligned16(dz) || !aligned16(Wp)) return MTGNN_EUNSUPPORTED;
  const PackLayout L(da, dm);
  const unsigned grid = (unsigned)cdiv(max_q, 16);
  TimedScope ts("merge_bwd", s);
  if (cdiv(da, 16) == 7)
    k_merge_bwd<7, 13><<<grid, 64 * MW, 0, s>>>(dz, Wp + L.off[3], Wp + L.off[4], Wp + L.off[5], m1, dm1, dm_in,
                                                dattn, n_q, max_q, da, dm);
  else
    k_merge_bwd<2, 4><<<grid, 64 * MW, 0, s>>>(dz, Wp + L.off[3], Wp + L.off[4], Wp + L.off[5], m1, dm1, dm_in,
                                               dattn, n_q, max_q, da, dm);
  MTGNN_CHECK_LAUNCH("merge_bwd");
  return MTGNN_OK;
}

}  // namespace mtgnn

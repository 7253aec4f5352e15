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

// Row tiles per block of the single-layer kernels (query projection, d M', GRU dx): one at a few thousand
// rows (two, half the weight-fragment loads per row, measured slower there: half the blocks), two from
// RT2_ROWS rows on, where the blocks far outnumber the CUs and the weight reads dominate.
constexpr int RT2_ROWS = 16384;
template <class F>
void with_row_tiles(int64_t rows, F f) {
  if (rows >= RT2_ROWS) f(std::integral_constant<int, 2>{});
  else f(std::integral_constant<int, 1>{});
}

template <int NCT> struct Tiles { static constexpr int per_wave = (NCT + MW - 1) / MW; };

// acc[r NU + u] (16 x 16 output tile t = wave + 4 u of row tile r) += X[16 rows of tile r, 16 KC]
// B[16 t.., 16 KC]^T.  X: the block's LDS tile of 16 RT rows (row stride XSS, zero beyond the true width).
// B: a zero-padded weight copy, 16 MW NU rows by 16 KC columns, so every fragment load is in bounds and
// unconditional; each fragment serves the RT row tiles.  PDT weight chunks are in flight ahead of the
// one being multiplied (PDT = KC: the whole share is requested at once, for launches too small to hide
// the latency with other blocks).
template <int NCT, int KC, int XSS = XS, int RT = 1, int PDT = PD>
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
  for (int c = 0; c < PDT && c < KC; ++c) load_b(c);
#pragma unroll
  for (int c = 0; c < KC; ++c) {
    if (c + PDT < KC) load_b(c + PDT);   // in flight while this chunk's MFMAs run
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
// (n <= XSS - col0; r0 < M).  Every load of a thread is issued before its first LDS store, so the tile costs
// one memory latency, not one per 64 MW elements: the loads are unconditional (a slot past the tile or past
// row M - 1 reads an element of the tile's last valid row and keeps zero), since a load under a per-lane
// condition is compiled into a branch of its own that waits for it.
template <int XSS = XS, int RT = 1, int NTH = 64 * MW>
__device__ __forceinline__ void load_rows(float* X, int col0, const float* __restrict__ src, int64_t ld, int n,
                                          int64_t r0, int64_t M) {
  constexpr int PER = (16 * RT * (XSS / 4) + NTH - 1) / NTH;
  const int nq = n / 4, tot = 16 * RT * nq;
  if (nq <= 0) return;
  const int64_t last = M - 1 - r0;   // >= 0: the tile's last valid row
  float4 v[PER];
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int e = threadIdx.x + NTH * k;
    const int ec = e < tot ? e : tot - 1;
    const int r = ec / nq, q = ec % nq;
    const bool ok = e < tot && r <= last;
    const float4 x = *reinterpret_cast<const float4*>(src + (r0 + (r <= last ? r : last)) * ld + 4 * q);
    v[k] = ok ? x : float4{0.f, 0.f, 0.f, 0.f};
  }
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int e = threadIdx.x + NTH * k;
    if (e < tot) *reinterpret_cast<float4*>(X + (e / nq) * XSS + col0 + 4 * (e % nq)) = v[k];
  }
}

template <int XSS = XS, int RT = 1, int NTH = 64 * MW>
__device__ __forceinline__ void zero_cols(float* X, int c0, int c1) {
  for (int e = threadIdx.x; e < 16 * RT * (c1 - c0); e += NTH)
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
constexpr int PREP_MAX = 18;   // the six merge copies and up to twelve extra copies
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
template <int NA, int KM, int RT>
__global__ __launch_bounds__(64 * MW) void k_qproj_fwd(const float* __restrict__ q_in, const float* __restrict__ Wp,
                                                       const float* __restrict__ cq, float* __restrict__ qv,
                                                       const int32_t* __restrict__ n_q, int64_t max_q, int da, int dm,
                                                       int Dq) {
  __shared__ __attribute__((aligned(16))) float X0[16 * RT * XS];
  const int64_t M = eff_count(max_q, n_q);
  const int64_t r0 = (int64_t)blockIdx.x * 16 * RT;
  if (r0 >= M) return;   // block-uniform
  zero_cols<XS, RT>(X0, dm, 16 * KM);
  load_rows<XS, RT>(X0, 0, q_in, Dq, dm, r0, M);
  __syncthreads();
  f32x4 acc[RT * Tiles<NA>::per_wave];
  layer<NA, KM, XS, RT>(X0, Wp, acc);
  each_out<NA, RT>(acc, da, r0, M, [&](int i, int j, bool ok, float v) {
    if (ok) qv[(r0 + i) * da + j] = v + cq[j];
  });
}

// dm_in[:, da:] += dqv W_q[:, :dm] (the memory part of the query input), WqT = W_q[:, :dm]^T padded.
template <int NM, int NA, int RT>
__global__ __launch_bounds__(64 * MW) void k_qproj_dx(const float* __restrict__ dqv, const float* __restrict__ WqT,
                                                      float* __restrict__ dm_in, int64_t ldm,
                                                      const int32_t* __restrict__ n_q, int64_t max_q, int da, int dm) {
  __shared__ __attribute__((aligned(16))) float X0[16 * RT * XS];
  const int64_t M = eff_count(max_q, n_q);
  const int64_t r0 = (int64_t)blockIdx.x * 16 * RT;
  if (r0 >= M) return;   // block-uniform
  zero_cols<XS, RT>(X0, da, 16 * NA);
  load_rows<XS, RT>(X0, 0, dqv, da, da, r0, M);
  __syncthreads();
  f32x4 acc[RT * Tiles<NM>::per_wave];
  layer<NM, NA, XS, RT>(X0, WqT, acc);
  each_out<NM, RT>(acc, dm, r0, M, [&](int i, int j, bool ok, float v) {
    if (ok) dm_in[(r0 + i) * ldm + da + j] += v;
  });
}

// d_mem[:, :dm] += S[:, dm : dm + 2 da] W_kv[:, :dm] over 16-row tiles (S: the per-row sums of
// [dh_q | dK | dV], row stride ldS; WkT = W_kv[:, :dm]^T padded).
template <int NM, int KK, int RT>
__global__ __launch_bounds__(64 * MW) void k_dmem_dx(const float* __restrict__ S, int64_t ldS,
                                                     const float* __restrict__ WkT, float* __restrict__ d_mem,
                                                     const int32_t* __restrict__ n_rows, int64_t max_rows, int dm,
                                                     int w2) {
  __shared__ __attribute__((aligned(16))) float X0[16 * RT * XS];
  const int64_t M = eff_count(max_rows, n_rows);
  const int64_t r0 = (int64_t)blockIdx.x * 16 * RT;
  if (r0 >= M) return;   // block-uniform
  zero_cols<XS, RT>(X0, w2, 16 * KK);
  load_rows<XS, RT>(X0, 0, S + dm, ldS, w2, r0, M);
  __syncthreads();
  f32x4 acc[RT * Tiles<NM>::per_wave];
  layer<NM, KK, XS, RT>(X0, WkT, acc);
  each_out<NM, RT>(acc, dm, r0, M, [&](int i, int j, bool ok, float v) {
    if (ok) d_mem[(r0 + i) * dm + j] += v;
  });
}

// The GRU backward's time-feature gradient: dmsg_time = dgi W_ih[:, c0 : c0 + dt] over 16-row tiles of dgi
// (3 dm wide); WT = W_ih[:, c0 : c0 + dt]^T zero-padded (gru_dx_weight_copy).
constexpr int XS_GRU = 308;   // >= 304 (19 chunks of 16), XS_GRU / 4 odd

template <int NT, int KC, int RT>
__global__ __launch_bounds__(64 * MW) void k_gru_dx(const float* __restrict__ dgi, int64_t ldg,
                                                    const float* __restrict__ WT, float* __restrict__ out, int dt,
                                                    const int32_t* __restrict__ n_rows, int64_t max_rows, int K) {
  __shared__ __attribute__((aligned(16))) float X0[16 * RT * XS_GRU];
  const int64_t M = eff_count(max_rows, n_rows);
  const int64_t r0 = (int64_t)blockIdx.x * 16 * RT;
  if (r0 >= M) return;   // block-uniform
  zero_cols<XS_GRU, RT>(X0, K, 16 * KC);
  load_rows<XS_GRU, RT>(X0, 0, dgi, ldg, K, r0, M);
  __syncthreads();
  f32x4 acc[RT * Tiles<NT>::per_wave];
  layer<NT, KC, XS_GRU, RT>(X0, WT, acc);
  each_out<NT, RT>(acc, dt, r0, M, [&](int i, int j, bool ok, float v) {
    if (ok) out[(r0 + i) * dt + j] = v;
  });
}

// ---------------------------------------------------------------- the GRU update on the layer machinery

// h is the message's first d_mem columns (h = M[node], the first slice of the message), so the reset and
// update gates' two products fold into one: W_ih,g x + W_hh,g h = (W_ih,g + [W_hh,g | 0]) x for g = r, z.
// Only the candidate gate keeps its hidden product apart (the reset gate multiplies it).
//
// A block owns 16 RT updated rows and U hidden units (unit group blockIdx.y).  Its output columns, packed
// in 16-wide tiles: TI tiles of the input product (the folded r columns, the folded z columns, the
// candidate's input columns: 3 U, zero-padded) over the KI message chunks, then TH tiles of the candidate's
// hidden product (U columns) over the KH chunks of h.  Job j (tile j of the TI + TH) goes to a wave in snake
// order (round j / NW left to right, the next round right to left), which balances the long input tiles
// against the short hidden ones; round q of a wave accumulates in acc[q].  The pre-activations meet in LDS
// and the gates are applied there.
constexpr int GRU_NW = 4;   // waves per block (eight measured no faster)
template <int NW>
struct GruJobs {
  static constexpr int job(int round, int wave) { return round * NW + ((round & 1) ? NW - 1 - wave : wave); }
};

// acc[q][r] += X (row tile r) B^T over the KC chunks, for the rounds q whose job lies in [JB, JE); the
// job's tile is tile (job - JB) of B, stored fragment-major: [JE - JB][KC][64 lanes][4] (fragment-major
// copy of a zero-padded [16 (JE - JB)][16 KC] matrix: lane l of chunk c holds row 16 t + l % 16, columns
// 16 c + 4 (l / 16) .. + 3).  The wave W is a template
// argument, so the rounds a wave skips cost no branch in the chunk loop (a branch there would make every
// chunk wait for all loads in flight, the prefetched ones included).
// `pre` runs once the first chunks' weight loads are in flight (the block's tile load, so that the two
// latencies overlap).
template <int NW, int NR, int KC, int XSS, int RT, int W, int JB, int JE, class Pre>
__device__ __forceinline__ void gru_jobs(const float* X, const float* __restrict__ B, f32x4 (&acc)[NR][RT], Pre pre) {
  const int lane = threadIdx.x & 63, fr = lane & 15, fg = lane >> 4;
  const float* Bl[NR];
#pragma unroll
  for (int q = 0; q < NR; ++q) {
    const int j = GruJobs<NW>::job(q, W);
    Bl[q] = B + (size_t)(j >= JB && j < JE ? j - JB : 0) * KC * 256 + 4 * lane;
  }
  float4 bf[KC][NR];
  auto load_b = [&](int c) {   // one contiguous 1 KB fragment per wave and tile
#pragma unroll
    for (int q = 0; q < NR; ++q)
      if (GruJobs<NW>::job(q, W) >= JB && GruJobs<NW>::job(q, W) < JE)
        bf[c][q] = *reinterpret_cast<const float4*>(Bl[q] + 256 * c);
  };
#pragma unroll
  for (int c = 0; c < PD && c < KC; ++c) load_b(c);
  pre();
#pragma unroll
  for (int c = 0; c < KC; ++c) {
    if (c + PD < KC) load_b(c + PD);
#pragma unroll
    for (int r = 0; r < RT; ++r) {
      const float4 a = *reinterpret_cast<const float4*>(X + (16 * r + fr) * XSS + 16 * c + 4 * fg);
#pragma unroll
      for (int q = 0; q < NR; ++q) {
        if (!(GruJobs<NW>::job(q, W) >= JB && GruJobs<NW>::job(q, W) < JE)) continue;
        f32x4& d = acc[q][r];
        d = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, bf[c][q].x, d, 0, 0, 0);
        d = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, bf[c][q].y, d, 0, 0, 0);
        d = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, bf[c][q].z, d, 0, 0, 0);
        d = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, bf[c][q].w, d, 0, 0, 0);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
  }
}

// The padded per-group weights (float32, fragment-major as gru_jobs reads them): Wi [S][16 TI][16 KI],
// Wh [S][16 TH][16 KH].  Row t of group g's
// Wi: t < U the folded reset row of unit g U + t, then U folded update rows, then U candidate input rows;
// row t < U of Wh: the candidate hidden row of unit g U + t.  Rows past those, units past d_mem and columns
// past the true width are zero.  Side job: the backward's padded W_ih time slice.
struct GruShape {
  int S, U, ti, th;
};
__global__ void k_gru_prepare(const float* __restrict__ W_ih, const float* __restrict__ W_hh, int dm, int dmsg,
                              int ki16, int kh16, GruShape sh, float* __restrict__ Wi, float* __restrict__ Wh,
                              GruWTArgs wt) {
  const int64_t e0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x, stride = (int64_t)gridDim.x * blockDim.x;
  const int64_t ni = (int64_t)sh.S * 16 * sh.ti * ki16, nh = (int64_t)sh.S * 16 * sh.th * kh16;
  for (int64_t x = e0; x < ni + nh; x += stride) {
    float v = 0.f;
    if (x < ni) {   // x = ((g ti + tile) KI + chunk) 256 + 4 lane + e
      const int rows = 16 * sh.ti;
      const int g = (int)(x / ((int64_t)rows * ki16)), w = (int)(x % ((int64_t)rows * ki16));
      const int tile = w / (16 * ki16), c = w / 256 % (ki16 / 16), l = w / 4 % 64, e = w % 4;
      const int t = 16 * tile + l % 16, col = 16 * c + 4 * (l / 16) + e;
      const int gate = t / sh.U, unit = sh.U * g + t % sh.U;
      if (gate < 3 && unit < dm && col < dmsg) {
        v = W_ih[(int64_t)(gate * dm + unit) * dmsg + col];
        if (gate < 2 && col < dm) v += W_hh[(int64_t)(gate * dm + unit) * dm + col];
      }
      Wi[x] = v;
    } else {
      const int64_t y = x - ni;
      const int rows = 16 * sh.th;
      const int g = (int)(y / ((int64_t)rows * kh16)), w = (int)(y % ((int64_t)rows * kh16));
      const int tile = w / (16 * kh16), c = w / 256 % (kh16 / 16), l = w / 4 % 64, e = w % 4;
      const int t = 16 * tile + l % 16, col = 16 * c + 4 * (l / 16) + e;
      const int unit = sh.U * g + t;
      if (t < sh.U && unit < dm && col < dm) v = W_hh[(int64_t)(2 * dm + unit) * dm + col];
      Wh[y] = v;
    }
  }
  if (wt.dst)
    for (int64_t x = e0; x < (int64_t)wt.rows * wt.cols; x += stride) {
      const int rr = (int)(x / wt.cols), cc = (int)(x % wt.cols);
      wt.dst[x] = (rr < wt.dt && cc < wt.K) ? W_ih[(int64_t)cc * wt.ld + wt.col0 + rr] : 0.f;
    }
}

template <int KI, int KH, int TI, int TH, int U, int RT, int NW>
__global__ __launch_bounds__(64 * NW) void k_gru_fused(const float* __restrict__ msg, int dmsg,
                                                       const float* __restrict__ Wi, const float* __restrict__ Wh,
                                                       const float* __restrict__ b_ih, const float* __restrict__ b_hh,
                                                       const int32_t* __restrict__ uniq,
                                                       const int32_t* __restrict__ winner, const float* __restrict__ t,
                                                       const int32_t* __restrict__ n_rows, int64_t max_rows, int dm,
                                                       float* __restrict__ mem, float* __restrict__ lu,
                                                       float* __restrict__ sr, float* __restrict__ sz,
                                                       float* __restrict__ sn, float* __restrict__ sghn) {
  constexpr int XL = 16 * KI + 4;          // LDS row strides, / 4 odd
  constexpr int GL = 16 * (TI + TH) + 4;
  constexpr int NR = (TI + TH + NW - 1) / NW;
  constexpr int NTH = 64 * NW;
  constexpr int ROWS = 16 * RT;
  constexpr int NB = 6 * U + 2 * ROWS;     // biases of the group's units (b_ih r, z, n, b_hh r, z, n), row ids
  constexpr int PB = (NB + NTH - 1) / NTH;
  __shared__ __attribute__((aligned(16))) float X[ROWS * XL];
  __shared__ float G[ROWS * GL];
  __shared__ float BS[6 * U];
  __shared__ int RI[2 * ROWS];             // node id, then the winning event, of each row
  const int64_t M = eff_count(max_rows, n_rows);
  const int64_t r0 = (int64_t)blockIdx.x * ROWS;
  if (r0 >= M) return;   // block-uniform
  const int g = blockIdx.y;
  const int lane = threadIdx.x & 63, fr = lane & 15, fg = lane >> 4;
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // the block's inputs: message rows, biases and row ids, all loads issued before the first LDS store
  auto prologue = [&]() {
    float bv[PB];
#pragma unroll
    for (int k = 0; k < PB; ++k) {
      const int e = threadIdx.x + NTH * k;
      bv[k] = 0.f;
      if (e < 6 * U) {
        const int unit = U * g + e % U, gate = e / U;
        if (unit < dm) bv[k] = (gate < 3 ? b_ih : b_hh)[(gate % 3) * dm + unit];
      } else if (e < NB) {
        const int i = (e - 6 * U) % ROWS;
        const int32_t* src = e - 6 * U < ROWS ? uniq : winner;
        bv[k] = __int_as_float(r0 + i < M ? src[r0 + i] : 0);
      }
    }
    zero_cols<XL, RT, NTH>(X, dmsg, 16 * KI);
    load_rows<XL, RT, NTH>(X, 0, msg, dmsg, dmsg, r0, M);
#pragma unroll
    for (int k = 0; k < PB; ++k) {
      const int e = threadIdx.x + NTH * k;
      if (e < 6 * U) BS[e] = bv[k];
      else if (e < NB) RI[e - 6 * U] = __float_as_int(bv[k]);
    }
    __syncthreads();
  };
  auto products = [&](auto wave) {
    constexpr int W = decltype(wave)::value;
    f32x4 acc[NR][RT];
#pragma unroll
    for (int q = 0; q < NR; ++q)
#pragma unroll
      for (int r = 0; r < RT; ++r) acc[q][r] = f32x4{0.f, 0.f, 0.f, 0.f};
    gru_jobs<NW, NR, KI, XL, RT, W, 0, TI>(X, Wi + (size_t)g * 16 * TI * 16 * KI, acc, prologue);
    gru_jobs<NW, NR, KH, XL, RT, W, TI, TI + TH>(X, Wh + (size_t)g * 16 * TH * 16 * KH, acc, [] {});
#pragma unroll
    for (int q = 0; q < NR; ++q) {
      const int j = GruJobs<NW>::job(q, W);
      if (j >= TI + TH) continue;
#pragma unroll
      for (int r = 0; r < RT; ++r)
#pragma unroll
        for (int e = 0; e < 4; ++e) G[(16 * r + 4 * fg + e) * GL + 16 * j + fr] = acc[q][r][e];
    }
  };
  // every wave runs the prologue (and its barrier) inside its own product body; the branch is wave-uniform
  static_assert(NW == 4 || NW == 8, "one product body per wave");
  switch (wid) {
    case 0: products(std::integral_constant<int, 0>{}); break;
    case 1: products(std::integral_constant<int, 1>{}); break;
    case 2: products(std::integral_constant<int, 2>{}); break;
    case 3: products(std::integral_constant<int, 3>{}); break;
    case 4: if constexpr (NW > 4) products(std::integral_constant<int, 4 % NW>{}); break;
    case 5: if constexpr (NW > 5) products(std::integral_constant<int, 5 % NW>{}); break;
    case 6: if constexpr (NW > 6) products(std::integral_constant<int, 6 % NW>{}); break;
    default: if constexpr (NW > 7) products(std::integral_constant<int, 7 % NW>{}); break;
  }
  __syncthreads();
  if (g == 0 && threadIdx.x < ROWS && r0 + threadIdx.x < M)   // last_update of the row's node
    lu[RI[threadIdx.x]] = t[RI[ROWS + threadIdx.x] >> 1];
  // gates: thread (row group rg, unit jj) takes rows rg, rg + RG, ...; its unit's biases stay in registers
  // and every LDS read of its rows is issued before the math
  constexpr int RG = NTH / U, PR = (ROWS + RG - 1) / RG;
  const int jj = threadIdx.x % U, rg = threadIdx.x / U, j = U * g + jj;
  if (rg >= RG || j >= dm) return;
  const float br = BS[jj] , bz = BS[U + jj], bn = BS[2 * U + jj];
  const float cr = BS[3 * U + jj], cz = BS[4 * U + jj], cn = BS[5 * U + jj];
  float pr[PR], pz[PR], pn[PR], ph[PR], hv[PR];
  int node[PR];
#pragma unroll
  for (int k = 0; k < PR; ++k) {
    const int i = rg + RG * k < ROWS ? rg + RG * k : ROWS - 1;
    const float* gi = G + i * GL;
    pr[k] = gi[jj];
    pz[k] = gi[U + jj];
    pn[k] = gi[2 * U + jj];
    ph[k] = gi[16 * TI + jj];
    hv[k] = X[i * XL + j];
    node[k] = RI[i];
  }
#pragma unroll
  for (int k = 0; k < PR; ++k) {
    const int i = rg + RG * k;
    if (i >= ROWS || r0 + i >= M) break;
    const float rr = sigmoid_hw((pr[k] + br) + cr);
    const float zz = sigmoid_hw((pz[k] + bz) + cz);
    const float ghn = ph[k] + cn;
    const float nn = tanh_hw((pn[k] + bn) + rr * ghn);
    const float hn = (1.f - zz) * nn + zz * hv[k];
    const int64_t row = r0 + i;
    mem[(int64_t)node[k] * dm + j] = hn;
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
    // z_src W_a, then z_dst and z_neg (adjacent LDS tiles) as two row tiles of one pass over W_b; every
    // weight chunk requested at once (a block per 16 targets: too few blocks to hide the latency)
    f32x4 as[NU], adn[2 * NU];
    layer<NA, NA, XL, 1, NA>(T[0], Wp, as);
    layer<NA, NA, XL, 2, NA>(T[1], Wp + WSZ, adn);
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      const int j = 16 * (wid + MW * u) + fr;
      if (j >= 16 * NA) continue;
      const float bj = j < da ? b1[j] : 0.f;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = 4 * fg + r;
        T[3][i * XL + j] = (as[u][r] + adn[u][r]) + bj;
        T[4][i * XL + j] = (as[u][r] + adn[NU + u][r]) + bj;
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
  // dz for the three query blocks: the sources through W_a^T, then destinations and negatives (adjacent
  // LDS tiles) as two row tiles of one pass over W_b^T
  {
    f32x4 acc[NU];
    layer<NA, NA, XL, 1, NA>(T[0], Wp + 2 * WSZ, acc);
    each_out<NA, 1>(acc, da, r0, n, [&](int i, int j, bool ok, float v) {
      if (ok) dz[(r0 + i) * da + j] = v;
    });
  }
  {
    f32x4 acc[2 * NU];
    layer<NA, NA, XL, 2, NA>(T[1], Wp + 3 * WSZ, acc);
#pragma unroll
    for (int b = 0; b < 2; ++b) {   // row tile b: query block 1 + b
      float* out = dz + (int64_t)(1 + b) * n * da;
#pragma unroll
      for (int u = 0; u < NU; ++u) {
        const int j = 16 * (wid + MW * u) + fr;
        if (j >= da) continue;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t row = r0 + 4 * fg + r;
          if (row < n) out[row * da + j] = acc[b * NU + u][r];
        }
      }
    }
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
  with_row_tiles(max_rows, [&](auto rt) {
    constexpr int RT = decltype(rt)::value;
    const unsigned grid = (unsigned)cdiv(max_rows, 16 * RT);
    if (cdiv(3 * dm, 16) == 19)
      k_gru_dx<7, 19, RT><<<grid, 64 * MW, 0, s>>>(dgi, 3 * dm, WT, dmsg_time, dt, n_rows, max_rows, 3 * dm);
    else
      k_gru_dx<2, 6, RT><<<grid, 64 * MW, 0, s>>>(dgi, 3 * dm, WT, dmsg_time, dt, n_rows, max_rows, 3 * dm);
  });
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
  with_row_tiles(max_rows, [&](auto rt) {
    constexpr int RT = decltype(rt)::value;
    const unsigned grid = (unsigned)cdiv(max_rows, 16 * RT);
    if (L.nm == 7)
      k_dmem_dx<7, 13, RT><<<grid, 64 * MW, 0, s>>>(S, ldS, Wp + L.off[2], d_mem, n_rows, max_rows, dm, 2 * da);
    else
      k_dmem_dx<2, 4, RT><<<grid, 64 * MW, 0, s>>>(S, ldS, Wp + L.off[2], d_mem, n_rows, max_rows, dm, 2 * da);
  });
  MTGNN_CHECK_LAUNCH("dmem_dx");
  return MTGNN_OK;
}

mtgnn_status qproj_fwd_fused(const float* q_in, const float* Wp, const float* cq, float* qv, const int32_t* n_q,
                             int64_t max_q, int da, int dm, int dt, hipStream_t s) {
  if (max_q <= 0) return MTGNN_OK;
  if (!aligned16(q_in) || !aligned16(Wp) || (dm + dt) % 4 != 0) return MTGNN_EUNSUPPORTED;
  const QLayout L(da, dm, dt);
  with_row_tiles(max_q, [&](auto rt) {
    constexpr int RT = decltype(rt)::value;
    const unsigned grid = (unsigned)cdiv(max_q, 16 * RT);
    if (L.na == 7)
      k_qproj_fwd<7, 7, RT><<<grid, 64 * MW, 0, s>>>(q_in, Wp + L.off[0], cq, qv, n_q, max_q, da, dm, dm + dt);
    else
      k_qproj_fwd<2, 2, RT><<<grid, 64 * MW, 0, s>>>(q_in, Wp + L.off[0], cq, qv, n_q, max_q, da, dm, dm + dt);
  });
  MTGNN_CHECK_LAUNCH("qproj_fwd");
  return MTGNN_OK;
}

mtgnn_status qproj_dx_fused(const float* dqv, const float* Wp, float* dm_in, int64_t ldm, const int32_t* n_q,
                            int64_t max_q, int da, int dm, int dt, hipStream_t s) {
  if (max_q <= 0) return MTGNN_OK;
  if (!aligned16(dqv) || !aligned16(Wp)) return MTGNN_EUNSUPPORTED;
  const QLayout L(da, dm, dt);
  with_row_tiles(max_q, [&](auto rt) {
    constexpr int RT = decltype(rt)::value;
    const unsigned grid = (unsigned)cdiv(max_q, 16 * RT);
    if (L.na == 7)
      k_qproj_dx<7, 7, RT><<<grid, 64 * MW, 0, s>>>(dqv, Wp + L.off[1], dm_in, ldm, n_q, max_q, da, dm);
    else
      k_qproj_dx<2, 2, RT><<<grid, 64 * MW, 0, s>>>(dqv, Wp + L.off[1], dm_in, ldm, n_q, max_q, da, dm);
  });
  MTGNN_CHECK_LAUNCH("qproj_dx");
  return MTGNN_OK;
}

// Unit groups: two for d_mem above 64 (more blocks at a few thousand rows), else one.  Rows per block:
// 32 from 16 Ki rows on (each weight fragment then serves two row tiles), else 16.
static bool gru_fused_shape(int dm, int dmsg, int& ki, int& kh, GruShape& sh) {
  ki = (int)cdiv(dmsg, 16);
  kh = (int)cdiv(dm, 16);
  sh.S = dm > 64 ? 2 : 1;
  sh.U = (int)cdiv(dm, sh.S);
  sh.ti = (int)cdiv(3 * sh.U, 16);
  sh.th = (int)cdiv(sh.U, 16);
  const bool wide = kh == 7 && sh.U == 50 && (ki == 19 || ki == 20 || ki == 30);   // ti 10, th 4
  const bool narrow = ki == 7 && kh == 2 && sh.U == 32;                               // ti 6, th 2
  return dm % 4 == 0 && dmsg % 4 == 0 && (wide || narrow);
}

bool gru_fused_ok(int dtype, int dm, int dmsg) {
  int ki, kh;
  GruShape sh;
  return dtype == MTGNN_F32 && gru_fused_shape(dm, dmsg, ki, kh, sh);
}

size_t gru_fused_weight_floats(int dm, int dmsg) {
  int ki, kh;
  GruShape sh;
  gru_fused_shape(dm, dmsg, ki, kh, sh);
  return (size_t)sh.S * 256 * ((size_t)sh.ti * ki + (size_t)sh.th * kh);
}

mtgnn_status gru_fused(const float* msg, const float* W_ih, const float* W_hh, const float* b_ih, const float* b_hh,
                       const int32_t* uniq, const int32_t* winner, const float* t, const int32_t* n_rows,
                       int64_t max_rows, int dm, int dmsg, float* Wp, float* mem, float* lu, float* sr, float* sz,
                       float* sn, float* sghn, GruWTArgs wt, hipStream_t s) {
  int ki, kh;
  GruShape sh;
  if (!gru_fused_shape(dm, dmsg, ki, kh, sh) || !aligned16(msg)) return MTGNN_EUNSUPPORTED;
  float* Wi = Wp;
  float* Wh = Wp + (size_t)sh.S * 256 * sh.ti * ki;
  const int64_t tot = (int64_t)gru_fused_weight_floats(dm, dmsg);
  k_gru_prepare<<<(unsigned)std::min<int64_t>(cdiv(tot, 256), 1024), 256, 0, s>>>(W_ih, W_hh, dm, dmsg, 16 * ki,
                                                                                   16 * kh, sh, Wi, Wh, wt);
  MTGNN_CHECK_LAUNCH("gru_prepare");
  if (max_rows <= 0) return MTGNN_OK;
  const int rt = max_rows >= 16384 ? 2 : 1;
  const dim3 grid((unsigned)cdiv(max_rows, 16 * rt), (unsigned)sh.S);
  TimedScope ts("gru_fused", s);
  auto launch = [&](auto kern) {
    kern<<<grid, 64 * GRU_NW, 0, s>>>(msg, dmsg, Wi, Wh, b_ih, b_hh, uniq, winner, t, n_rows, max_rows, dm, mem,
                                         lu, sr, sz, sn, sghn);
  };
  if (ki == 19) {
    if (rt == 2) launch(k_gru_fused<19, 7, 10, 4, 50, 2, GRU_NW>);
    else launch(k_gru_fused<19, 7, 10, 4, 50, 1, GRU_NW>);
  } else if (ki == 20) {
    if (rt == 2) launch(k_gru_fused<20, 7, 10, 4, 50, 2, GRU_NW>);
    else launch(k_gru_fused<20, 7, 10, 4, 50, 1, GRU_NW>);
  } else if (ki == 30) {
    if (rt == 2) launch(k_gru_fused<30, 7, 10, 4, 50, 2, GRU_NW>);
    else launch(k_gru_fused<30, 7, 10, 4, 50, 1, GRU_NW>);
  } else {
    if (rt == 2) launch(k_gru_fused<7, 2, 6, 2, 32, 2, GRU_NW>);
    else launch(k_gru_fused<7, 2, 6, 2, 32, 1, GRU_NW>);
  }
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

int link_pad_copies(const float* W1, int da, float* Wp, PadCopy* out) {
  if (!link_fused_ok(da) || !aligned16(Wp)) return 0;
  const int na = (int)cdiv(da, 16);
  const int rows = 16 * MW * (int)cdiv(na, MW), cols = 16 * na;
  const size_t wsz = (size_t)rows * cols;
  // zero-padded W_a, W_b (the column halves of W_d1) and their transposes
  for (int m = 0; m < 4; ++m)
    out[m] = PadCopy{W1 + (m % 2 ? da : 0), Wp + m * wsz, rows, cols, da, da, 2 * da, m >= 2 ? 1 : 0, cols};
  return 4;
}

mtgnn_status pad_copies(const PadCopy* c, int n, hipStream_t s) {
  if (n < 0 || n > PREP_MAX) return MTGNN_EINVAL;
  if (n == 0) return MTGNN_OK;
  PrepArgs a;
  int64_t most = 0;
  for (int m = 0; m < n; ++m) {
    a.src[m] = c[m].src;
    a.dst[m] = c[m].dst;
    a.rows[m] = c[m].rows;
    a.cols[m] = c[m].cols;
    a.n[m] = c[m].n;
    a.k[m] = c[m].k;
    a.ld[m] = c[m].ld;
    a.tr[m] = c[m].tr;
    a.ldd[m] = c[m].ldd > 0 ? c[m].ldd : c[m].cols;
    most = std::max<int64_t>(most, (int64_t)c[m].rows * c[m].cols);
  }
  a.ncopy = n;
  k_merge_prepare<<<dim3((unsigned)cdiv(most, 256), (unsigned)n), 256, 0, s>>>(a);
  MTGNN_CHECK_LAUNCH("pad_copies");
  return MTGNN_OK;
}

mtgnn_status link_prepare_weights(const float* W1, int da, float* Wp, hipStream_t s) {
  PadCopy c[4];
  if (link_pad_copies(W1, da, Wp, c) != 4) return MTGNN_EUNSUPPORTED;
  return pad_copies(c, 4, s);
}

mtgnn_status link_fused(const float* z, const int32_t* n_q, int64_t max_q, int da, const float* W1, const float* b1,
                        const float* W2, const float* b2, float* Wp, float* DA, float* DB, float* part, float* dz,
                        float* scores, float* dW2, float* db2, float* loss, hipStream_t s, bool prepared,
                        bool s_reduce) {
  if (!link_fused_ok(da) || !aligned16(z) || !aligned16(Wp) || !aligned16(dz)) return MTGNN_EUNSUPPORTED;
  if (!prepared) MTGNN_TRY(link_prepare_weights(W1, da, Wp, s));
  const int na = (int)cdiv(da, 16);
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
  return s_reduce ? MTGNN_OK : link_reduce(part, n_q, max_q, da, dW2, db2, loss, s);
}

mtgnn_status link_reduce(const float* part, const int32_t* n_q, int64_t max_q, int da, float* dW2, float* db2,
                         float* loss, hipStream_t s) {
  // blocks past the device's target count wrote no partial: sum only those below it
  k_link_reduce_dev<<<(unsigned)cdiv(da + 2, 4), 256, 0, s>>>(part, n_q, max_q / 3, da, dW2, db2, loss);
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

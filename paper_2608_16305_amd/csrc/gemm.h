// Strided fp32-accumulating MFMA "strip" GEMM for gfx950:  C(i,j) = sum_k A(i,k) B(k,j).
//
// A(i,k) = A[i*a_si + k*a_sk], B(k,j) = B[k*b_sk + j*b_sj], C row-major.
// One template covers the three products of a linear layer y = x W^T + b:
//   forward   y  = x  W^T : A = x (k-contiguous),         B(k,j) = W[j][k] (k-contiguous)
//   data grad dx = dy W   : A = dy (k-contiguous),        B(k,j) = W[k][j] (j-contiguous)
//   weight    dW = dy^T x : A(i,k) = dy[k][i] (i-contig.), B(k,j) = x[k][j] (j-contiguous)
//
// Shape: the layer widths here are 32..500, while the row counts (events,
// queries, neighbour slots) are 10^3..10^7.  A block therefore owns a strip of
// 64 rows and up to 256 columns (the whole output width in one strip for
// widths <= 256), so each A element is read from HBM once.  Each of the 4
// waves computes 16 rows x BN columns with v_mfma_f32_16x16x4_f32 (lane l
// supplies A[l%16][l/16] and B[l/16][l%16]; accumulator register r of lane l
// is C[4*(l/16)+r][l%16]).  Operands move global -> registers -> LDS in
// 32-deep k steps with 4-wide loads along each operand's contiguous
// dimension; LDS keeps both operands k-contiguous and double-buffered (one
// barrier per k step), so every MFMA operand comes from a 16-byte LDS read.
// Inputs may be float32 or bfloat16 (converted on load).
#pragma once

#include <algorithm>
#include <type_traits>

#include "common.h"

namespace mtgnn {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));

// Four float32 values as the bfloat16 operand of an MFMA (k = 4 (l / 16) .. + 3 of lane l, in order).
// Weights stored as bfloat16 are exact in float32: their high halves are taken as they are.
__device__ __forceinline__ s16x4 bf16x4_exact(float4 v) {
  const uint32_t lo = (__float_as_uint(v.x) >> 16) | (__float_as_uint(v.y) & 0xffff0000u);
  const uint32_t hi = (__float_as_uint(v.z) >> 16) | (__float_as_uint(v.w) & 0xffff0000u);
  s16x4 r;
  r.x = (short)(lo & 0xffffu);
  r.y = (short)(lo >> 16);
  r.z = (short)(hi & 0xffffu);
  r.w = (short)(hi >> 16);
  return r;
}
// Activations are rounded to bfloat16 (nearest, ties to even) as they enter a bfloat16 product; values
// already rounded by their producer pass through unchanged.
__device__ __forceinline__ s16x4 bf16x4_round(float4 v) {
  auto rn = [](float f) {
    const uint32_t u = __float_as_uint(f);
    return (short)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
  };
  s16x4 r;
  r.x = rn(v.x);
  r.y = rn(v.y);
  r.z = rn(v.z);
  r.w = rn(v.w);
  return r;
}

// Call-site tags: the hot sites get their own kernel symbol (and timer name).
namespace site {
struct Generic { static constexpr const char* name = "gemm"; };
struct KvProj { static constexpr const char* name = "gemm_kv_proj"; };    // K, V = kv_in W^T + b (neighbour slots)
struct KvDw { static constexpr const char* name = "gemm_kv_dw"; };        // dW_k, dW_v (+ db) over neighbour slots
struct KvDx { static constexpr const char* name = "gemm_kv_dx"; };        // dphi = dK W_k,t + dV W_v,t
struct GruDw { static constexpr const char* name = "gemm_gru_dw"; };      // dW_ih, dW_hh (+ biases) over updated rows
}  // namespace site

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
  int ksplit_dev = 0;          // > 0: split z covers the z-th of ksplit_dev equal chunks (multiples of 16) of the
                               // device count K_dev instead (every split holds rows whatever the count)
  int64_t c_split_stride;      // element offset of split z's output
  const float* gate;           // optional: result *= (gate(i,j) > 0)  (ReLU backward)
  int64_t ldgate;
  int round_bf16;              // round the stored result to bfloat16 (kept as float32)
  int a_vec = 0, b_vec = 0;    // 4-wide loads along the contiguous dimension are aligned (set by the launcher)
  int64_t ones_col = -1;       // B column treated as all ones (-1: none); its results go to col_out
  float* col_out = nullptr;    // C(i, ones_col) is written to col_out[i] (weight-grad GEMMs: the bias grad)
  int xcd_group = 1;           // place blocks that share an operand chunk on one XCD (see gemm_tile)
  // Time-encoder gradient epilogue: instead of writing C, each block writes the
  // column sums over its rows of  g = -C(i,j) sin(arg_ij)  and of  g * delta_i
  // (arg_ij = w_j delta_i + b_j) to tg_part[row block][0 / 1][j].
  float* tg_part = nullptr;
  const float* tg_sin = nullptr;     // saved sin(arg) [M, N] (row stride N), or null: recomputed
  const float* tg_delta = nullptr;   // per-row delta_i, or null: 0
  const float* tg_w = nullptr;       // time encoder w, b (used when tg_sin is null)
  const float* tg_b = nullptr;
  int tile_bn = 0;             // host-side plan: output tile width (0: chosen by gemm_tile_width)
  int tile_bk = 16;            // host-side plan: k step (64 only for weight-gradient 64-wide tiles)
};

// Tile coordinates of this block.  Workgroups are dispatched round-robin over
// the 8 XCDs (block L runs on XCD L mod 8), and each XCD has its own L2.  The
// blocks that read the same operand chunk form a group: with split-K, the
// blocks of one k-chunk (they all read the same rows of the row-indexed
// operand); otherwise the column strips of one row block (same A rows).
// Group q is placed on XCD q mod 8, so a group's blocks share that XCD's L2,
// and consecutive groups still spread over every XCD (a device-side row count
// that leaves only the first groups active keeps all XCDs busy).  Groups past
// the last multiple of 8 keep the plain order.
struct TileCoord {
  int64_t x, y, z;
};
__device__ __forceinline__ TileCoord gemm_tile(int xcd_group) {
  const uint32_t gx = gridDim.x, gy = gridDim.y, gz = gridDim.z;
  const uint32_t L = blockIdx.x + gx * (blockIdx.y + gy * blockIdx.z);
  uint32_t V = L;
  const uint32_t G = gz > 1 ? gx * gy : gy;       // blocks per group
  const uint32_t ngroups = gz > 1 ? gz : gx;
  const uint32_t full = G * (ngroups & ~7u);
  if (xcd_group && G > 1 && L < full) {
    const uint32_t xcd = L & 7u, slot = L >> 3;
    V = (xcd + 8u * (slot / G)) * G + slot % G;
  }
  TileCoord t;
  if (gz > 1) {   // V = (z * gx + x) * gy + y
    t.y = V % gy;
    t.x = (V / gy) % gx;
    t.z = V / (gy * gx);
  } else {        // V = x * gy + y
    t.y = V % gy;
    t.x = V / gy;
    t.z = 0;
  }
  return t;
}

// Epilogue rounding of a float32 value to the nearest bfloat16 (ties to even), widened back.
__device__ __forceinline__ float round_to_bf16(float v) { return bf16_to_f32(f32_to_bf16(v)); }

constexpr int G_BK = 16, G_THREADS = 256;   // BK: k step of the library's launches (split-K chunks are multiples)

// Four consecutive elements as float (fp32: one 16-byte load; bf16: one 8-byte load).
template <typename T>
struct Vec4;
template <>
struct Vec4<float> {
  __device__ __forceinline__ static float4 load(const float* p) { return *reinterpret_cast<const float4*>(p); }
};
template <>
struct Vec4<uint16_t> {
  __device__ __forceinline__ static float4 load(const uint16_t* p) {
    const uint2 u = *reinterpret_cast<const uint2*>(p);
    return float4{bf16_to_f32((uint16_t)(u.x & 0xffffu)), bf16_to_f32((uint16_t)(u.x >> 16)),
                  bf16_to_f32((uint16_t)(u.y & 0xffffu)), bf16_to_f32((uint16_t)(u.y >> 16))};
  }
};

// LDS layout of one operand tile (R rows of an output dimension x BK of the
// reduction).  Operands contiguous along k are stored k-contiguous, [R][BK+4]:
// a lane's four values of a 16-deep chunk come from one 16-byte read.  Operands
// contiguous along their rows are stored as loaded, [BK][R+pad], with pad
// chosen so consecutive k rows sit 16 banks apart; their fragment is four
// 4-byte reads.  Either way, sub-step s of chunk kc gives lane l the value at
// k = kc + 4 (l/16) + s.
template <bool KC, int R, int BK>
struct Lds {
  static constexpr int LDK = BK + 4;                          // KC row stride
  // Row-contiguous row stride, == 4 mod 32: a fragment read takes k = kc + 4 (l/16) + i, so the two lane
  // groups of a 32-lane half are 4 LDR apart, which is then 16 banks (with LDR == 16 mod 32 it was 0
  // banks: a 2-way conflict on every read).
  static constexpr int LDR = R + ((4 - (R % 32)) + 32) % 32;
  static constexpr int SIZE = KC ? R * LDK : BK * LDR;
  __device__ __forceinline__ static float4 frag(const float* lds, int row, int kc, int lane) {
    const int k = kc + 4 * (lane >> 4);
    if (KC) return *reinterpret_cast<const float4*>(lds + row * LDK + k);
    return float4{lds[(k + 0) * LDR + row], lds[(k + 1) * LDR + row], lds[(k + 2) * LDR + row],
                  lds[(k + 3) * LDR + row]};
  }
  // group of 4: along k (KC) at (mn, k..k+3), or along rows at (mn..mn+3, k)
  __device__ __forceinline__ static void put(float* lds, int mn, int k, float4 v) {
    if (KC) *reinterpret_cast<float4*>(lds + mn * LDK + k) = v;
    else *reinterpret_cast<float4*>(lds + k * LDR + mn) = v;
  }
  __device__ __forceinline__ static void coord(int g, int& mn, int& k) {
    if (KC) { mn = g / (BK / 4); k = (g % (BK / 4)) * 4; }
    else { mn = (g % (R / 4)) * 4; k = g / (R / 4); }
  }
};

// One operand tile moving global -> registers -> LDS, for any shape: 4-wide
// loads where a group is in range and aligned (vec), element loads otherwise.
template <typename T, bool KC, int R, int BK>
struct TileIO {
  using L = Lds<KC, R, BK>;
  static constexpr int GROUPS = R * BK / 4;
  static constexpr int PER = (GROUPS + G_THREADS - 1) / G_THREADS;
  float4 v[PER];

  // e(mn, k) = base[mn * s_mn + k * s_k]; rows < rows_lim and k < k_lim are in range
  __device__ __forceinline__ void load(const T* base, int64_t s_mn, int64_t s_k, int64_t mn0, int64_t k0,
                                       int64_t rows_lim, int64_t k_lim, bool vec, int64_t ones_mn, int tid) {
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int g = tid + p * G_THREADS;
      float e[4] = {0.f, 0.f, 0.f, 0.f};
      if (g < GROUPS) {
        int mn, k;
        L::coord(g, mn, k);
        const int64_t gm = mn0 + mn, gk = k0 + k;
        const bool full = KC ? (gm < rows_lim && gk + 3 < k_lim) : (gm + 3 < rows_lim && gk < k_lim);
        const bool has_ones = ones_mn >= gm && ones_mn <= (KC ? gm : gm + 3);   // virtual column: no memory
        if (vec && full && !has_ones) {
          const float4 f = Vec4<T>::load(base + gm * s_mn + gk * s_k);
          e[0] = f.x; e[1] = f.y; e[2] = f.z; e[3] = f.w;
        } else {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int64_t m = KC ? gm : gm + i, kk = KC ? gk + i : gk;
            if (m < rows_lim && kk < k_lim) e[i] = m == ones_mn ? 1.f : Elem<T>::load(base, m * s_mn + kk * s_k);
          }
        }
      }
      v[p] = float4{e[0], e[1], e[2], e[3]};
    }
  }

  __device__ __forceinline__ void store(float* lds, int tid) const {
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int g = tid + p * G_THREADS;
      if (g >= GROUPS) continue;
      int mn, k;
      L::coord(g, mn, k);
      L::put(lds, mn, k, v[p]);
    }
  }
};

// Branch-free variant of TileIO for aligned shapes (every row count of the
// operand's contiguous dimension and every k extent are multiples of 4).  Each
// thread keeps a pointer per 4-wide group and advances it by a constant per k
// step; groups outside the matrix load from its first element (a valid
// address) and are zeroed by selects, so the loop has no per-element branches.
template <typename T, bool KC, int R, int BK>
struct TileVec {
  using L = Lds<KC, R, BK>;
  static constexpr int GROUPS = R * BK / 4;
  static constexpr int PER = (GROUPS + G_THREADS - 1) / G_THREADS;
  const T* ptr[PER];
  const T* safe;
  int kq[PER];          // k offset of the group inside the tile
  uint32_t row_ok;      // bit p: the group's rows exist
  uint32_t ones;        // bit p: the group holds the virtual all-ones column (value 1 in its first row)
  float4 v[PER];

  __device__ __forceinline__ void init(const T* base, int64_t s_mn, int64_t s_k, int64_t mn0, int64_t k0,
                                       int64_t rows_lim, int64_t ones_mn, int tid) {
    safe = base;
    row_ok = 0;
    ones = 0;
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int g = tid + p * G_THREADS;
      int mn, k;
      L::coord(g, mn, k);
      const int64_t gm = mn0 + mn;
      const bool is_ones = !KC && gm == ones_mn;
      const bool ok = g < GROUPS && gm < rows_lim && !is_ones;
      if (ok) row_ok |= 1u << p;
      if (g < GROUPS && is_ones) ones |= 1u << p;
      kq[p] = k;
      ptr[p] = base + (ok ? gm : 0) * s_mn + (k0 + k) * s_k;
    }
  }
  // k0: first k of the tile; k_lim: end of the reduction range
  __device__ __forceinline__ void load_into(int64_t k0, int64_t k_lim, float4* dst) const {
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const bool kin = k0 + kq[p] < k_lim;
      const bool ok = ((row_ok >> p) & 1u) && kin;
      const float4 f = Vec4<T>::load(ok ? ptr[p] : safe);
      const bool one = ((ones >> p) & 1u) && kin;
      dst[p] = float4{ok ? f.x : (one ? 1.f : 0.f), ok ? f.y : 0.f, ok ? f.z : 0.f, ok ? f.w : 0.f};
    }
  }
  __device__ __forceinline__ void load(int64_t k0, int64_t k_lim) { load_into(k0, k_lim, v); }
  __device__ __forceinline__ void advance(int64_t step) {
#pragma unroll
    for (int p = 0; p < PER; ++p) ptr[p] += step;
  }
  __device__ __forceinline__ void store_from(float* lds, int tid, const float4* src) const {
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int g = tid + p * G_THREADS;
      if (g >= GROUPS) continue;
      int mn, k;
      L::coord(g, mn, k);
      L::put(lds, mn, k, src[p]);
    }
  }
  __device__ __forceinline__ void store(float* lds, int tid) const { store_from(lds, tid, v); }
};

// Time-gradient epilogue of a (64 WM)-row block (4 waves x WM 16-row tiles): instead of C,
// write the column sums over the block's rows of  g = -C(i,j) sin(arg_ij)  and of
// g * delta_i to tg_part[row block][0 / 1][j].  red: 8 BN floats of LDS that no
// wave reads any more.
template <int BN, int WM>
__device__ __forceinline__ void gemm_store_timegrad(const GemmArgs& g, const TileCoord tc, int64_t M,
                                                    const f32x4 (&acc)[WM][BN / 16], float* red) {
  constexpr int NT = BN / 16;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int64_t row0 = tc.x * 64 * WM, col0 = tc.y * BN;
  float* red_w = red;
  float* red_b = red + 4 * BN;
#pragma unroll
  for (int j = 0; j < NT; ++j) {
    const int64_t gj = col0 + j * 16 + (lane & 15);
    float cw = 0.f, cb = 0.f;
    if (gj < g.N) {
#pragma unroll
      for (int i = 0; i < WM; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t gi = row0 + (wid * WM + i) * 16 + 4 * (lane >> 4) + r;
        if (gi >= M) continue;
        const float d = g.tg_delta ? g.tg_delta[gi] : 0.f;
        const float sn = g.tg_sin ? g.tg_sin[gi * g.N + gj] : sinf(time_arg(g.tg_w[gj], d, g.tg_b[gj]));
        const float gv = acc[i][j][r] * -sn;
        cb += gv;
        cw += gv * d;
      }
    }
    cw += __shfl_xor(cw, 16, 64);
    cb += __shfl_xor(cb, 16, 64);
    cw += __shfl_xor(cw, 32, 64);
    cb += __shfl_xor(cb, 32, 64);
    if (lane < 16) {
      red_w[wid * BN + j * 16 + lane] = cw;
      red_b[wid * BN + j * 16 + lane] = cb;
    }
  }
  __syncthreads();
  for (int c = tid; c < BN; c += G_THREADS) {
    const int64_t gj = col0 + c;
    if (gj >= g.N) continue;
    g.tg_part[(tc.x * 2 + 0) * g.N + gj] = ((red_w[c] + red_w[BN + c]) + red_w[2 * BN + c]) + red_w[3 * BN + c];
    g.tg_part[(tc.x * 2 + 1) * g.N + gj] = ((red_b[c] + red_b[BN + c]) + red_b[2 * BN + c]) + red_b[3 * BN + c];
  }
}

// Epilogue of a (64 WM) x BN block: bias, accumulate, ReLU gate / pre-activation,
// bf16 rounding, bias-grad column, split-K partial placement.
template <int BN, int WM>
__device__ __forceinline__ void gemm_store(const GemmArgs& g, const TileCoord tc, int64_t M,
                                           const f32x4 (&acc)[WM][BN / 16]) {
  constexpr int NT = BN / 16;
  constexpr int BM = 64 * WM;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int64_t row0 = tc.x * BM, col0 = tc.y * BN;
  float* C = g.C + tc.z * g.c_split_stride;
  const bool split = g.c_split_stride != 0;
#pragma unroll
  for (int j = 0; j < NT; ++j) {
    const int64_t gj = col0 + j * 16 + (lane & 15);
    if (gj >= g.N) continue;
    const bool to_col = gj == g.ones_col && !split;
    const float bj = g.bias ? g.bias[gj] : 0.f;
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t gi = row0 + (wid * WM + i) * 16 + 4 * (lane >> 4) + r;
        if (gi >= M) continue;
        float v = acc[i][j][r] + bj;
        if (g.accumulate) v += C[gi * g.ldc + gj];
        if (g.gate && !(g.gate[gi * g.ldgate + gj] > 0.f)) v = 0.f;
        if (g.relu) {
          g.C2[gi * g.ldc2 + gj] = v;
          v = fmaxf(v, 0.f);
        }
        if (g.round_bf16) v = round_to_bf16(v);
        if (to_col) g.col_out[gi] = v;
        else C[gi * g.ldc + gj] = v;
      }
  }
}

// Block: (64 WM) rows x BN columns; wave w computes WM 16-row tiles x BN.
// Within each 16-deep k chunk, lane l feeds the MFMA k-slot l/16 with
// k = 4 (l/16) + s at sub-step s (s = 0..3), for both operands (see Lds); the
// sum over the chunk is unchanged.  NBUF = 2: double-buffered LDS, one barrier per k step; NBUF = 1:
// one LDS buffer, the next tile waits in registers (two barriers per step).
// VEC: aligned shapes use the branch-free TileVec loader.
template <class Site, int BN, int WM, int BK, int NBUF, bool VEC, typename TA, typename TB, bool A_KCONTIG,
          bool B_KCONTIG, int PF = 1, bool TGE = false>
__device__ __forceinline__ void gemm_body(const GemmArgs& g, const TileCoord tc) {
  constexpr int NT = BN / 16;
  constexpr int BM = 64 * WM;
  using LA = Lds<A_KCONTIG, BM, BK>;
  using LB = Lds<B_KCONTIG, BN, BK>;
  __shared__ float As[NBUF][LA::SIZE];
  __shared__ float Bs[NBUF][LB::SIZE];

  const int64_t M = eff_count(g.M, g.M_dev);
  const int64_t Kall = eff_count(g.K, g.K_dev);
  const int64_t row0 = tc.x * BM;
  const int64_t col0 = tc.y * BN;
  if (row0 >= M) return;
  const int64_t kchunk = g.ksplit_dev > 0 ? cdiv(cdiv(Kall, g.ksplit_dev), 16) * 16 : g.kchunk;
  const int64_t kbeg = tc.z * kchunk;
  const int64_t kend = min(Kall, kbeg + kchunk);

  const TA* A = (const TA*)g.A;
  const TB* B = (const TB*)g.B;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int64_t a_smn = g.a_si, a_sk = g.a_sk, b_smn = g.b_sj, b_sk = g.b_sk;

  f32x4 acc[WM][NT];
#pragma unroll
  for (int i = 0; i < WM; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  using IOA = typename std::conditional<VEC, TileVec<TA, A_KCONTIG, BM, BK>, TileIO<TA, A_KCONTIG, BM, BK>>::type;
  using IOB = typename std::conditional<VEC, TileVec<TB, B_KCONTIG, BN, BK>, TileIO<TB, B_KCONTIG, BN, BK>>::type;
  IOA ta;
  IOB tb;
  auto load_tiles = [&](int64_t k0) {
    if constexpr (VEC) {
      ta.load(k0, kend);
      tb.load(k0, kend);
      ta.advance(BK * a_sk);
      tb.advance(BK * b_sk);
    } else {
      ta.load(A, a_smn, a_sk, row0, k0, M, kend, g.a_vec != 0, -1, tid);
      tb.load(B, b_smn, b_sk, col0, k0, g.N, kend, g.b_vec != 0, g.ones_col, tid);
    }
  };

  // Forward products with bfloat16 weights (x W^T, both operands contiguous along k) run on the bfloat16
  // MFMA: the activations enter rounded to bfloat16 (they already are: every forward input of the
  // bfloat16 mode is stored or produced rounded), products are exact and accumulate in float32.
  constexpr bool MMA_BF16 = std::is_same<TB, uint16_t>::value && A_KCONTIG && B_KCONTIG && !TGE;

  // MFMA work on one LDS tile pair
  auto compute = [&](const float* as, const float* bs) {
#pragma unroll
    for (int kc = 0; kc < BK; kc += 16) {
      float4 a4[WM];
#pragma unroll
      for (int i = 0; i < WM; ++i) a4[i] = LA::frag(as, (wid * WM + i) * 16 + (lane & 15), kc, lane);
      float4 b4[NT];
#pragma unroll
      for (int j = 0; j < NT; ++j) b4[j] = LB::frag(bs, j * 16 + (lane & 15), kc, lane);
      if constexpr (MMA_BF16) {   // one 16 x 16 x 16 bfloat16 MFMA per tile pair and chunk
        s16x4 ab[WM], bb[NT];
#pragma unroll
        for (int i = 0; i < WM; ++i) ab[i] = bf16x4_round(a4[i]);
#pragma unroll
        for (int j = 0; j < NT; ++j) bb[j] = bf16x4_exact(b4[j]);
#pragma unroll
        for (int i = 0; i < WM; ++i)
#pragma unroll
          for (int j = 0; j < NT; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(ab[i], bb[j], acc[i][j], 0, 0, 0);
        continue;
      }
#pragma unroll
      for (int i = 0; i < WM; ++i)
#pragma unroll
        for (int j = 0; j < NT; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4[i].x, b4[j].x, acc[i][j], 0, 0, 0);
#pragma unroll
      for (int i = 0; i < WM; ++i)
#pragma unroll
        for (int j = 0; j < NT; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4[i].y, b4[j].y, acc[i][j], 0, 0, 0);
#pragma unroll
      for (int i = 0; i < WM; ++i)
#pragma unroll
        for (int j = 0; j < NT; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4[i].z, b4[j].z, acc[i][j], 0, 0, 0);
#pragma unroll
      for (int i = 0; i < WM; ++i)
#pragma unroll
        for (int j = 0; j < NT; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4[i].w, b4[j].w, acc[i][j], 0, 0, 0);
    }
  };

  if constexpr (VEC && PF == 2 && NBUF == 2) {
    // Prefetch distance 2: register sets 0 and 1 alternate (the loop is
    // unrolled by two so each set stays in fixed registers).  While tile t is
    // computed from LDS buffer t % 2, tile t + 2 is loading into the register
    // set that held tile t, and tile t + 1 (loaded one iteration earlier) is
    // then written to the other LDS buffer.
    if (kbeg < kend) {
      float4 ra0[IOA::PER], rb0[IOB::PER], ra1[IOA::PER], rb1[IOB::PER];
      const int64_t ntile = cdiv(kend - kbeg, BK);
      ta.init(A, a_smn, a_sk, row0, kbeg, M, -1, tid);
      tb.init(B, b_smn, b_sk, col0, kbeg, g.N, g.ones_col, tid);
      auto fetch = [&](int64_t t, float4* ra, float4* rb) {
        ta.load_into(kbeg + t * BK, kend, ra);
        tb.load_into(kbeg + t * BK, kend, rb);
        ta.advance(BK * a_sk);
        tb.advance(BK * b_sk);
      };
      fetch(0, ra0, rb0);
      if (ntile > 1) fetch(1, ra1, rb1);
      ta.store_from(As[0], tid, ra0);
      tb.store_from(Bs[0], tid, rb0);
      __syncthreads();
      for (int64_t t = 0; t < ntile; t += 2) {
        if (t + 2 < ntile) fetch(t + 2, ra0, rb0);
        compute(As[0], Bs[0]);
        if (t + 1 < ntile) {
          ta.store_from(As[1], tid, ra1);
          tb.store_from(Bs[1], tid, rb1);
        }
        __syncthreads();
        if (t + 1 >= ntile) break;
        if (t + 3 < ntile) fetch(t + 3, ra1, rb1);
        compute(As[1], Bs[1]);
        if (t + 2 < ntile) {
          ta.store_from(As[0], tid, ra0);
          tb.store_from(Bs[0], tid, rb0);
        }
        __syncthreads();
      }
    }
  } else if (kbeg < kend) {
    if constexpr (VEC) {
      ta.init(A, a_smn, a_sk, row0, kbeg, M, -1, tid);
      tb.init(B, b_smn, b_sk, col0, kbeg, g.N, g.ones_col, tid);
    }
    load_tiles(kbeg);
    ta.store(As[0], tid);
    tb.store(Bs[0], tid);
    __syncthreads();
    int cur = 0;
    for (int64_t k0 = kbeg; k0 < kend; k0 += BK) {
      const bool more = k0 + BK < kend;
      if (more) load_tiles(k0 + BK);
      compute(As[cur], Bs[cur]);
      if (more) {
        const int nb = NBUF == 2 ? (cur ^ 1) : 0;
        if (NBUF == 1) __syncthreads();   // every wave is done reading the only buffer
        ta.store(As[nb], tid);
        tb.store(Bs[nb], tid);
      }
      __syncthreads();
      if (NBUF == 2) cur ^= 1;
    }
  }

  if constexpr (TGE) {   // time-gradient epilogue (tg_* arguments)
    static_assert(8 * BN <= NBUF * LA::SIZE, "time-gradient epilogue scratch");
    gemm_store_timegrad<BN, WM>(g, tc, M, acc, &As[0][0]);   // the operand tiles are no longer read
    return;
  }
  gemm_store<BN, WM>(g, tc, M, acc);
}

// One output tile per block; tile coordinates from the XCD-grouped order.
template <class Site, int BN, int WM, int BK, int NBUF, bool VEC, typename TA, typename TB, bool A_KCONTIG,
          bool B_KCONTIG, int PF = 1, bool TGE = false>
__global__ __launch_bounds__(G_THREADS) void k_gemm(GemmArgs g) {
  gemm_body<Site, BN, WM, BK, NBUF, VEC, TA, TB, A_KCONTIG, B_KCONTIG, PF, TGE>(g, gemm_tile(g.xcd_group));
}

// Up to G_MAXBATCH independent products of one shape class in one launch:
// blockIdx.z = problem * zper + split.  Blocks beyond a problem's own column
// strips or splits return at once.
constexpr int G_MAXBATCH = 4;
struct GemmBatch {
  GemmArgs a[G_MAXBATCH];
  int n;
  int zper;
};

template <class Site, int BN, int WM, int BK, int NBUF, bool VEC, typename TA, typename TB, bool A_KCONTIG,
          bool B_KCONTIG>
__global__ __launch_bounds__(G_THREADS) void k_gemm_batch(GemmBatch b) {
  const int p = (int)(blockIdx.z / (uint32_t)b.zper);
  if (p >= b.n) return;
  const GemmArgs& g = b.a[p];
  TileCoord tc;
  tc.x = blockIdx.x;
  tc.y = blockIdx.y;
  tc.z = blockIdx.z % (uint32_t)b.zper;
  if (tc.y * BN >= g.N || (g.ksplit_dev == 0 && tc.z * g.kchunk >= g.K)) return;
  gemm_body<Site, BN, WM, BK, NBUF, VEC, TA, TB, A_KCONTIG, B_KCONTIG>(g, tc);
}

// Tile shape used by the library's launches.
constexpr int G_WM = 1, G_NBUF = 2;
// Row tiles per wave of the time-gradient products (64-row blocks; 128-row blocks, with half the
// weight-strip reads and partial sums, measured slower on the neighbour-slot product: 60 vs 52 us).
constexpr int G_WM_TG = 1;
constexpr int G_TG_ROWS = 64 * G_WM_TG;   // rows per partial of a time-gradient product

// Column `ones_col` (if >= 0) goes to col_out[i] instead of out.
__global__ void k_splitk_reduce(const float* __restrict__ part, int64_t split_stride, int nsplit, int64_t rows,
                                int64_t cols, float* __restrict__ out, int64_t ldo, int64_t ones_col,
                                float* __restrict__ col_out);
// The same, with rows from row_split on written to out_hi / col_out_hi (row index minus row_split).
__global__ void k_splitk_reduce_rows2(const float* __restrict__ part, int64_t split_stride, int nsplit, int64_t rows,
                                      int64_t cols, float* __restrict__ out, float* __restrict__ out_hi, int64_t ldo,
                                      int64_t ones_col, float* __restrict__ col_out, float* __restrict__ col_out_hi,
                                      int64_t row_split);

// Strip width for an output of N columns: equal strips of at most 128 columns
// (32, 64, 112 or 128 wide).  Narrower strips need less LDS, so more blocks
// share a CU; that measured faster than reading the A rows once.
int gemm_strip_width(int64_t N);
// Weight gradients over many rows: one strip up to 256 columns (64 .. 256 wide).
int gemm_wide_strip_width(int64_t N);
// Tile width for an M x N output: full strips, or 32-wide tiles when strips would
// leave the launch with few blocks (small row counts are latency-bound; more,
// narrower blocks put more waves on each SIMD).
int gemm_tile_width(int64_t M, int64_t N, int ksplit);
// Weight-gradient plan over R reduction rows for an N x K output.
struct DwPlan {
  int ksplit;
  int64_t kchunk;
  int bn, bk;
  int ksplit_dev = 0;   // > 0: the splits cut the device row count (GemmArgs::ksplit_dev)
};
DwPlan dw_plan(int64_t R, int64_t N, int64_t K);
// With a device row count, `tiles` output tiles per split: the splits cut the device count into
// equal chunks, so every split holds rows, with about DW_DEV_BLOCKS blocks in all and never more
// splits than the host plan (whose workspace then suffices).
constexpr int64_t DW_DEV_BLOCKS = 512;
DwPlan dw_plan_dev(DwPlan host, int64_t tiles);

// A 4-wide load along the contiguous dimension is aligned when the base and the other stride are.
inline bool vec_ok(const void* p, int64_t other_stride, size_t esz) {
  return ((uintptr_t)p % (4 * esz)) == 0 && (other_stride % 4) == 0;
}

template <class Site, int BN, bool VEC, typename TA, typename TB, bool AK, bool BK, int KSTEP = G_BK,
          bool TGE = false>
void gemm_kernel_launch(const GemmArgs& g, dim3 grid, hipStream_t s) {
  k_gemm<Site, BN, TGE ? G_WM_TG : G_WM, KSTEP, G_NBUF, VEC, TA, TB, AK, BK, 1, TGE><<<grid, G_THREADS, 0, s>>>(g);
}

template <class Site, bool VEC, typename TA, typename TB, bool AK, bool BK>
void gemm_bn_launch(const GemmArgs& g, int bn, dim3 grid, hipStream_t s) {
  if constexpr (AK && !BK) {   // data gradients: the time-gradient epilogue
    if (g.tg_part != nullptr) {
      switch (bn) {
        case 32: gemm_kernel_launch<Site, 32, VEC, TA, TB, AK, BK, G_BK, true>(g, grid, s); break;
        case 64: gemm_kernel_launch<Site, 64, VEC, TA, TB, AK, BK, G_BK, true>(g, grid, s); break;
        case 112: gemm_kernel_launch<Site, 112, VEC, TA, TB, AK, BK, G_BK, true>(g, grid, s); break;
        default: gemm_kernel_launch<Site, 128, VEC, TA, TB, AK, BK, G_BK, true>(g, grid, s); break;
      }
      return;
    }
  }
  if constexpr (AK || BK) {   // forward and data-gradient products: strips of at most 128 columns
    switch (bn) {
      case 32: gemm_kernel_launch<Site, 32, VEC, TA, TB, AK, BK>(g, grid, s); break;
      case 64: gemm_kernel_launch<Site, 64, VEC, TA, TB, AK, BK>(g, grid, s); break;
      case 112: gemm_kernel_launch<Site, 112, VEC, TA, TB, AK, BK>(g, grid, s); break;
      default: gemm_kernel_launch<Site, 128, VEC, TA, TB, AK, BK>(g, grid, s); break;
    }
    return;
  }
  switch (bn) {
    case 32: gemm_kernel_launch<Site, 32, VEC, TA, TB, AK, BK>(g, grid, s); break;
    case 112: gemm_kernel_launch<Site, 112, VEC, TA, TB, AK, BK>(g, grid, s); break;
    case 64:
      if constexpr (!AK && !BK) {   // weight gradients: 64-deep k steps on 64 x 64 tiles
        if (g.tile_bk == 64) {
          gemm_kernel_launch<Site, 64, VEC, TA, TB, AK, BK, 64>(g, grid, s);
          break;
        }
      }
      gemm_kernel_launch<Site, 64, VEC, TA, TB, AK, BK>(g, grid, s);
      break;
    case 128: gemm_kernel_launch<Site, 128, VEC, TA, TB, AK, BK>(g, grid, s); break;
    case 160: gemm_kernel_launch<Site, 160, VEC, TA, TB, AK, BK>(g, grid, s); break;
    case 208: gemm_kernel_launch<Site, 208, VEC, TA, TB, AK, BK>(g, grid, s); break;
    default: gemm_kernel_launch<Site, 256, VEC, TA, TB, AK, BK>(g, grid, s); break;
  }
}

// The branch-free loader needs 4-aligned bases and strides, row counts of
// each operand's contiguous dimension that are multiples of 4, a virtual
// ones column (if any) at a multiple of 4, and k extents (host K and the
// split chunk) that are multiples of 4 for operands contiguous along k.
template <typename TA, typename TB, bool AK, bool BK>
bool gemm_vec_ok(const GemmArgs& g) {
  return vec_ok(g.A, AK ? g.a_si : g.a_sk, sizeof(TA)) && vec_ok(g.B, BK ? g.b_sj : g.b_sk, sizeof(TB)) &&
         (AK ? (g.K % 4 == 0 && g.kchunk % 4 == 0 && g.K_dev == nullptr) : (g.M % 4 == 0 && g.M_dev == nullptr)) &&
         (BK ? (g.K % 4 == 0 && g.kchunk % 4 == 0 && g.K_dev == nullptr) : g.N % 4 == 0 || g.ones_col == g.N - 1) &&
         (g.ones_col < 0 || g.ones_col % 4 == 0);
}
template <typename TA, typename TB, bool AK, bool BK>
void gemm_set_vec_flags(GemmArgs& g) {   // general loader: 4-wide only when aligned
  g.a_vec = vec_ok(g.A, AK ? g.a_si : g.a_sk, sizeof(TA)) ? 1 : 0;
  g.b_vec = vec_ok(g.B, BK ? g.b_sj : g.b_sk, sizeof(TB)) ? 1 : 0;
}

bool gemm_rs_applicable(const GemmArgs& g);
mtgnn_status gemm_rs_launch(const GemmArgs& g, hipStream_t s, bool bf16_weights = false);

template <class Site, typename TA, typename TB, bool AK, bool BK>
mtgnn_status gemm_launch_t(const GemmArgs& g0, int ksplit, hipStream_t s) {
  if constexpr (std::is_same<Site, site::KvProj>::value && std::is_same<TA, float>::value && AK && BK) {
    // key/value projection over the neighbour slots: weight-stationary kernel (gemm_rs.h), with float32 or
    // bfloat16 weights (the slot rows are float32 holding bfloat16 values in that mode)
    if (ksplit <= 1 && gemm_rs_applicable(g0)) {
      TimedScope ts(Site::name, s);
      return gemm_rs_launch(g0, s, std::is_same<TB, uint16_t>::value);
    }
  }
  GemmArgs g = g0;
  gemm_set_vec_flags<TA, TB, AK, BK>(g);
  const int bn = g.tile_bn > 0 ? g.tile_bn : gemm_tile_width(g.M, g.N, ksplit);
  const int64_t bm = (AK && !BK && g.tg_part != nullptr) ? G_TG_ROWS : 64 * G_WM;   // time-gradient form: taller
  dim3 grid((unsigned)cdiv(g.M, bm), (unsigned)cdiv(g.N, bn), (unsigned)(ksplit < 1 ? 1 : ksplit));
  const bool vec = gemm_vec_ok<TA, TB, AK, BK>(g);
  TimedScope ts(Site::name, s);
  if (vec) gemm_bn_launch<Site, true, TA, TB, AK, BK>(g, bn, grid, s);
  else gemm_bn_launch<Site, false, TA, TB, AK, BK>(g, bn, grid, s);
  MTGNN_CHECK_LAUNCH(Site::name);
  return MTGNN_OK;
}

template <class Site, int BN, bool VEC, typename TA, typename TB, bool AK, bool BK>
void gemm_batch_kernel(const GemmBatch& b, dim3 grid, hipStream_t s) {
  if constexpr (!AK && !BK && BN == 64) {   // weight gradients on 64-wide tiles may take 64-deep steps
    if (b.a[0].tile_bk == 64) {
      k_gemm_batch<Site, BN, G_WM, 64, G_NBUF, VEC, TA, TB, AK, BK><<<grid, G_THREADS, 0, s>>>(b);
      return;
    }
  }
  k_gemm_batch<Site, BN, G_WM, G_BK, G_NBUF, VEC, TA, TB, AK, BK><<<grid, G_THREADS, 0, s>>>(b);
}

// Batched launch: every problem shares the tile width of the first (its tile_bn, or the width rule
// at its shape) and the launch uses the branch-free loader only if every problem allows it.
template <class Site, typename TA, typename TB, bool AK, bool BK>
mtgnn_status gemm_batch_launch_t(const GemmArgs* gs, int n, int zper, hipStream_t s) {
  if (n < 1 || n > G_MAXBATCH || zper < 1) return MTGNN_EINVAL;
  GemmBatch b{};
  b.n = n;
  b.zper = zper;
  const int bn = gs[0].tile_bn > 0 ? gs[0].tile_bn : gemm_tile_width(gs[0].M, gs[0].N, zper);
  bool vec = true;
  int64_t gx = 1, gy = 1;
  for (int i = 0; i < n; ++i) {
    b.a[i] = gs[i];
    gemm_set_vec_flags<TA, TB, AK, BK>(b.a[i]);
    vec = vec && gemm_vec_ok<TA, TB, AK, BK>(b.a[i]);
    gx = std::max<int64_t>(gx, cdiv(gs[i].M, 64 * G_WM));
    gy = std::max<int64_t>(gy, cdiv(gs[i].N, bn));
  }
  dim3 grid((unsigned)gx, (unsigned)gy, (unsigned)(n * zper));
  TimedScope ts(Site::name, s);
#define MTGNN_BATCH_BN(W)                                                    \
  case W:                                                                    \
    if (vec) gemm_batch_kernel<Site, W, true, TA, TB, AK, BK>(b, grid, s);   \
    else gemm_batch_kernel<Site, W, false, TA, TB, AK, BK>(b, grid, s);      \
    break;
  if constexpr (AK || BK) {
    switch (bn) {
      MTGNN_BATCH_BN(32)
      MTGNN_BATCH_BN(64)
      MTGNN_BATCH_BN(112)
      default:
        if (vec) gemm_batch_kernel<Site, 128, true, TA, TB, AK, BK>(b, grid, s);
        else gemm_batch_kernel<Site, 128, false, TA, TB, AK, BK>(b, grid, s);
        break;
    }
  } else {
    switch (bn) {
      MTGNN_BATCH_BN(32)
      MTGNN_BATCH_BN(64)
      MTGNN_BATCH_BN(112)
      MTGNN_BATCH_BN(128)
      MTGNN_BATCH_BN(160)
      MTGNN_BATCH_BN(208)
      default:
        if (vec) gemm_batch_kernel<Site, 256, true, TA, TB, AK, BK>(b, grid, s);
        else gemm_batch_kernel<Site, 256, false, TA, TB, AK, BK>(b, grid, s);
        break;
    }
  }
#undef MTGNN_BATCH_BN
  MTGNN_CHECK_LAUNCH(Site::name);
  return MTGNN_OK;
}

template <class Site, bool AK, bool BK>
mtgnn_status gemm_batch_launch(const GemmArgs* gs, int n, int zper, int dtype_a, int dtype_b, hipStream_t s) {
  if (dtype_a == MTGNN_F32 && dtype_b == MTGNN_F32) return gemm_batch_launch_t<Site, float, float, AK, BK>(gs, n, zper, s);
  if (dtype_a == MTGNN_F32) return gemm_batch_launch_t<Site, float, uint16_t, AK, BK>(gs, n, zper, s);
  if (dtype_b == MTGNN_F32) return MTGNN_EUNSUPPORTED;
  return gemm_batch_launch_t<Site, uint16_t, uint16_t, AK, BK>(gs, n, zper, s);
}

template <class Site, bool AK, bool BK>
mtgnn_status gemm_launch(const GemmArgs& g, int dtype_a, int dtype_b, int ksplit, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return MTGNN_OK;
  if (dtype_a == MTGNN_F32 && dtype_b == MTGNN_F32) return gemm_launch_t<Site, float, float, AK, BK>(g, ksplit, s);
  if (dtype_a == MTGNN_F32) return gemm_launch_t<Site, float, uint16_t, AK, BK>(g, ksplit, s);
  if (dtype_b == MTGNN_F32) return MTGNN_EUNSUPPORTED;   // bf16 activations always meet bf16 weights
  return gemm_launch_t<Site, uint16_t, uint16_t, AK, BK>(g, ksplit, s);
}

// The instances the library uses, each compiled in one place: gemm_nt.hip (x W^T, both operands
// contiguous along k), gemm_nn.hip (dy W) and gemm_tn.hip (dy^T x).  One translation unit per operand
// layout: each takes one to two minutes to compile, and the build runs them in parallel.
#define MTGNN_GEMM_INSTANCES(EXTERN)                                                                                 \
  EXTERN template mtgnn_status gemm_launch<site::Generic, true, true>(const GemmArgs&, int, int, int, hipStream_t);  \
  EXTERN template mtgnn_status gemm_launch<site::KvProj, true, true>(const GemmArgs&, int, int, int, hipStream_t);   \
  EXTERN template mtgnn_status gemm_batch_launch<site::Generic, true, true>(const GemmArgs*, int, int, int, int,      \
                                                                            hipStream_t);
#define MTGNN_GEMM_INSTANCES_NN(EXTERN)                                                                              \
  EXTERN template mtgnn_status gemm_launch<site::Generic, true, false>(const GemmArgs&, int, int, int, hipStream_t); \
  EXTERN template mtgnn_status gemm_launch<site::KvDx, true, false>(const GemmArgs&, int, int, int, hipStream_t);
#define MTGNN_GEMM_INSTANCES_TN(EXTERN)                                                                              \
  EXTERN template mtgnn_status gemm_launch<site::Generic, false, false>(const GemmArgs&, int, int, int, hipStream_t); \
  EXTERN template mtgnn_status gemm_launch<site::KvDw, false, false>(const GemmArgs&, int, int, int, hipStream_t);   \
  EXTERN template mtgnn_status gemm_batch_launch<site::Generic, false, false>(const GemmArgs*, int, int, int, int,    \
                                                                              hipStream_t);                          \
  EXTERN template mtgnn_status gemm_batch_launch<site::GruDw, false, false>(const GemmArgs*, int, int, int, int,      \
                                                                            hipStream_t);
MTGNN_GEMM_INSTANCES(extern)
MTGNN_GEMM_INSTANCES_NN(extern)
MTGNN_GEMM_INSTANCES_TN(extern)

// y[M,N] (+)= x[M,K] W[N,K]^T + bias.
// pre_relu: store the pre-activation there and relu(y) in y.  round_bf16: round y to bfloat16.
template <class Site = site::Generic>
mtgnn_status linear_fwd(const void* x, int x_dtype, int64_t ldx, const void* W, int w_dtype, int64_t ldw,
                        const float* bias, float* y, int64_t ldy, int64_t M, const int32_t* M_dev, int64_t N,
                        int64_t K, bool accumulate, hipStream_t s, float* pre_relu = nullptr, int64_t ldpre = 0,
                        bool round_bf16 = false) {
  GemmArgs g{};
  g.M = M; g.N = N; g.K = K; g.M_dev = M_dev;
  g.A = x; g.a_si = ldx; g.a_sk = 1;
  g.B = W; g.b_sk = 1; g.b_sj = ldw;
  g.C = y; g.ldc = ldy; g.bias = bias; g.accumulate = accumulate ? 1 : 0;
  g.relu = pre_relu ? 1 : 0; g.C2 = pre_relu; g.ldc2 = ldpre;
  g.kchunk = K; g.c_split_stride = 0; g.round_bf16 = round_bf16 ? 1 : 0;
  return gemm_launch<Site, true, true>(g, x_dtype, w_dtype, 1, s);
}

// dx[M,K] (+)= dy[M,N] W[N,K]; gate: dx *= (gate > 0) elementwise (after accumulation)
template <class Site = site::Generic>
mtgnn_status linear_dx(const float* dy, int64_t lddy, const void* W, int w_dtype, int64_t ldw, float* dx,
                       int64_t lddx, int64_t M, const int32_t* M_dev, int64_t N, int64_t K, bool accumulate,
                       hipStream_t s, const float* gate = nullptr, int64_t ldgate = 0) {
  GemmArgs g{};
  g.M = M; g.N = K; g.K = N; g.M_dev = M_dev;
  g.A = dy; g.a_si = lddy; g.a_sk = 1;
  g.B = W; g.b_sk = ldw; g.b_sj = 1;
  g.C = dx; g.ldc = lddx; g.accumulate = accumulate ? 1 : 0;
  g.kchunk = N; g.c_split_stride = 0; g.gate = gate; g.ldgate = ldgate;
  return gemm_launch<Site, true, false>(g, MTGNN_F32, w_dtype, 1, s);
}

// Time-gradient form of linear_dx: dphi = dy W is not stored; each G_TG_ROWS-row block
// writes its column sums of -dphi sin(arg) (and times delta) to part[block][2][K].
// Rows come from M (clamped by M_dev); part needs gemm_tg_blocks(M) * 2 * K floats.
inline int64_t gemm_tg_blocks(int64_t M) { return cdiv(M < 1 ? 1 : M, G_TG_ROWS); }
template <class Site = site::Generic>
mtgnn_status linear_dx_timegrad(const float* dy, int64_t lddy, const void* W, int w_dtype, int64_t ldw, int64_t M,
                                const int32_t* M_dev, int64_t N, int64_t K, const float* sin_saved,
                                const float* delta, const float* tw, const float* tb, float* part, hipStream_t s) {
  GemmArgs g{};
  g.M = M; g.N = K; g.K = N; g.M_dev = M_dev;
  g.A = dy; g.a_si = lddy; g.a_sk = 1;
  g.B = W; g.b_sk = ldw; g.b_sj = 1;
  g.C = nullptr; g.ldc = 0;
  g.kchunk = N; g.c_split_stride = 0;
  g.tg_part = part; g.tg_sin = sin_saved; g.tg_delta = delta; g.tg_w = tw; g.tg_b = tb;
  g.tile_bn = gemm_tile_width(M, K, 1);
  return gemm_launch<Site, true, false>(g, MTGNN_F32, w_dtype, 1, s);
}

// dW[N,K] = dy[R,N]^T x[R,K], reduction over R rows (clamped by R_dev), split-K through ws.
// db (optional): db[N] = sum over rows of dy, computed as an extra all-ones column of x.
size_t linear_dw_ws_bytes(int64_t R, int64_t N, int64_t K);

bool dw_rs_applicable(const float* X, int64_t ldx, int nx, const void* Y, int y_dtype, int64_t ldy, int ny);
mtgnn_status dw_rs_launch(const float* X, int64_t ldx, int nx, const float* Y, int64_t ldy, int ny, int64_t R,
                          const int32_t* R_dev, float* dW, int64_t lddw, float* db, void* ws, size_t ws_bytes,
                          hipStream_t s);
// The same, with output rows from row_split on written to dW_hi / db_hi.
mtgnn_status dw_rs_launch_rows2(const float* X, int64_t ldx, int nx, const float* Y, int64_t ldy, int ny, int64_t R,
                                const int32_t* R_dev, float* dW, float* dW_hi, int64_t lddw, float* db, float* db_hi,
                                int row_split, void* ws, size_t ws_bytes, hipStream_t s);

template <class Site = site::Generic>
mtgnn_status linear_dw(const float* dy, int64_t lddy, const void* x, int x_dtype, int64_t ldx, float* dW,
                       int64_t lddw, int64_t R, const int32_t* R_dev, int64_t N, int64_t K, void* ws,
                       size_t ws_bytes, hipStream_t s, float* db = nullptr) {
  if constexpr (std::is_same<Site, site::KvDw>::value) {
    // key/value weight gradient over the neighbour slots: output-stationary kernel (gemm_rs.h)
    if (db && dw_rs_applicable(dy, lddy, (int)N, x, x_dtype, ldx, (int)K))
      return dw_rs_launch(dy, lddy, (int)N, (const float*)x, ldx, (int)K, R, R_dev, dW, lddw, db, ws, ws_bytes, s);
  }
  const int64_t Kc = db ? K + 1 : K;   // extra all-ones column of x gives the bias gradient
  DwPlan plan = dw_plan(R, N, Kc);
  if (R_dev) plan = dw_plan_dev(plan, cdiv(N, 64 * G_WM) * cdiv(Kc, plan.bn));
  const int ksplit = plan.ksplit;
  const int64_t kchunk = plan.kchunk;
  GemmArgs g{};
  g.tile_bn = plan.bn;
  g.tile_bk = plan.bk;
  g.ksplit_dev = plan.ksplit_dev;
  g.M = N; g.N = Kc; g.K = R; g.K_dev = R_dev;
  if (db) { g.ones_col = K; g.col_out = db; }
  g.A = dy; g.a_si = 1; g.a_sk = lddy;
  g.B = x; g.b_sk = ldx; g.b_sj = 1;
  g.kchunk = kchunk;
  if (ksplit == 1) {
    g.C = dW; g.ldc = lddw; g.c_split_stride = 0;
    return gemm_launch<Site, false, false>(g, MTGNN_F32, x_dtype, 1, s);
  }
  if (ws_bytes < linear_dw_ws_bytes(R, N, K)) return MTGNN_EWORKSPACE;
  g.C = (float*)ws; g.ldc = Kc; g.c_split_stride = N * Kc;
  MTGNN_TRY((gemm_launch<Site, false, false>(g, MTGNN_F32, x_dtype, ksplit, s)));
  const int64_t tot = N * Kc;
  k_splitk_reduce<<<(unsigned)cdiv(tot, 64), 256, 0, s>>>((const float*)ws, N * Kc, ksplit, N, Kc, dW, lddw,
                                                           db ? K : -1, db);
  MTGNN_CHECK_LAUNCH("splitk_reduce");
  return MTGNN_OK;
}

// ---------------------------------------------------------------- batched products

// Independent forward products over the same rows M (clamped by M_dev):
// y_i[M, N_i] = x_i[M, K_i] W_i[N_i, K_i]^T + b_i, in one launch.
struct FwdProblem {
  const void* x;
  int64_t ldx;
  const void* W;
  int64_t ldw;
  const float* bias;
  float* y;
  int64_t ldy;
  int64_t N, K;
};
mtgnn_status linear_fwd_batch(const FwdProblem* ps, int n, int64_t M, const int32_t* M_dev, int x_dtype,
                              int w_dtype, hipStream_t s);

// Independent weight gradients over the same reduction rows R (clamped by R_dev):
// dW_i[N_i, K_i] = dy_i[R, N_i]^T x_i[R, K_i], and db_i = column sums of dy_i when db_i is set.
// One product launch and one split-K reduce launch for the whole batch.
struct DwProblem {
  const float* dy;
  int64_t lddy;
  const void* x;
  int64_t ldx;
  float* dW;
  int64_t lddw;
  int64_t N, K;
  float* db;
  // Optional (row_den > 0): dy is zero outside rows [R row_lo / row_den, R row_hi / row_den) of the R rows (the
  // device count), so the output-stationary kernel skips the rest (the strip kernel sums them all).
  int row_lo = 0, row_hi = 0, row_den = 0;
};
size_t linear_dw_batch_ws_bytes(int64_t R, const int64_t* N, const int64_t* K, int n);   // sizes only

// Batched output-stationary weight gradients (gemm_rs.h), for float32 outputs of at
// most 7 x 13 16 x 16 tiles: part_p[block][nx_p][ny_p + 1] = X_p^T [Y_p | 1] over the
// blocks' 16-row chunks.  Problem p owns blocks b_begin .. b_begin + nblk - 1.
struct DwOsProblem {
  const float* X;
  int64_t ldx;
  const float* Y;
  int64_t ldy;
  float* part;
  int nx, ny, b_begin, nblk;
  int row_lo = 0, row_hi = 0, row_den = 0;   // row_den > 0: only rows [R lo / den, R hi / den) of the R can be nonzero
};
constexpr int DW_OS_MAXP = 16;   // problems (or output tiles) per launch
struct DwOsBatch {
  DwOsProblem p[DW_OS_MAXP];
  int n;
  int64_t R;
  const int32_t* R_dev;
};
constexpr int DW_OS_MAX_BLOCKS = 256;
template <class Site = site::Generic>
mtgnn_status dw_os_launch(const DwOsBatch& b, int grid, hipStream_t s);
int dw_os_cu_count();

// A weight gradient cut into output tiles for the output-stationary kernel: tile t is
// dW_t[nx, ny] = X_t^T Y_t and, if db, db_t[nx] = column sums of X_t, over the R rows (clamped by R_dev);
// X_t, Y_t start at the tile's first column (row strides ldx, ldy; 16-byte aligned, strides multiples of
// 4), nx and ny multiples of 4 with nx <= 112 and ny <= 108.  Rows i < dup_rows of the tile's output are
// also written to dup (row stride lddup; if not null) and, with db, their sums to dup_db (if not null):
// a product that another weight shares.
struct DwTile {
  const float* X;
  int64_t ldx;
  const float* Y;
  int64_t ldy;
  int nx, ny;
  float* dW;
  int64_t lddw;
  float* db;
  float* dup;
  int64_t lddup;
  int dup_rows;
  float* dup_db;
};
size_t dw_tiles_ws_bytes(const DwTile* t, int n);
template <class Site = site::Generic>
mtgnn_status dw_tiles(const DwTile* t, int n, int64_t R, const int32_t* R_dev, void* ws, size_t ws_bytes,
                      hipStream_t s);
template <class Site = site::Generic>
mtgnn_status linear_dw_batch(const DwProblem* ps, int n, int64_t R, const int32_t* R_dev, int x_dtype, void* ws,
                             size_t ws_bytes, hipStream_t s);

}  // namespace mtgnn

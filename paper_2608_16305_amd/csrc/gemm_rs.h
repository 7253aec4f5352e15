// Weight-stationary fp32 MFMA product for many rows and a small second operand:
//   C(i,j) = sum_k A[i*a_si + k] B(k,j) (+ bias_j),   B(k,j) = B[k*b_sk + j*b_sj],
// with K <= 256 and ceil(N/16) >= 4 column tiles.  Used for the neighbour-slot
// products, whose row count (valid slots) is 10^4..10^7 while B is one layer's
// weight (about 200 x 200).
//
// Each of the 4 waves of a block keeps its share of B in registers for the
// whole launch: NTW = floor(NCT/4) full 16-column tiles (all of K), plus, for
// each of the NR = NCT mod 4 remaining column tiles, the k chunks c with
// c mod 4 = wave.  A block is persistent: it walks 16-row tiles of A (tile
// b, b + grid, ...), each brought into LDS by global_load_lds_dwordx4 one tile
// ahead (two slots, one barrier per tile).  Per tile every wave multiplies the
// 16 A rows by its register tiles and stores them; the remainder tiles'
// four k-partials go to LDS and are summed in wave order by one wave at the
// next tile (the summing wave rotates with the tile, so work stays balanced).
//
// MFMA v_mfma_f32_16x16x4_f32: lane l supplies A[row l%16][k] and B[k][col l%16]
// with k = 16 c + 4 (l/16) + s at sub-step s of chunk c, and holds
// C[4 (l/16) + r][l%16] in accumulator register r.
//
// LDS: A slot rows have a stride of KS floats (KS/4 odd, KS >= 16 KC), so the
// 16 rows of a fragment read hit distinct banks; positions K .. 16 KC of each
// row are zero.  LDS is only touched through inline assembly with explicit waits
// (lds_dma.h).  Global stores never need to be
// waited for: the DMA wait is vmcnt(0) with the next tile's load issued a full
// tile earlier.
#pragma once

#include "lds_dma.h"

namespace mtgnn {

namespace rs {

constexpr int stride_for(int kc) {   // smallest stride >= 16 kc floats with stride / 4 odd
  return (16 * kc / 4) % 2 == 1 ? 16 * kc : 16 * kc + 4;
}

}  // namespace rs

// Grid: blocks of 256 threads; block b handles row tiles b, b + gridDim.x, ...
// Requirements (checked by gemm_rs_ok on the host): A 16-byte aligned, a_sk = 1,
// a_si % 4 == 0, K % 4 == 0, 16 (KC - 1) < K <= 16 KC <= 256, N <= 16 NCT.
template <class Site, int NCT, int KC, int OCC>
__global__ __launch_bounds__(G_THREADS, OCC) void k_gemm_rs(GemmArgs g) {
  constexpr int NTW = NCT / 4, NR = NCT % 4;
  constexpr int KQ = (KC + 3) / 4;                 // remainder chunks per wave, at most
  constexpr int KS = rs::stride_for(KC);           // A row stride in LDS (floats)
  constexpr int SLOT = 16 * KS;                    // floats per A slot
  constexpr int RED = NR * 4 * 64 * 4;             // floats per parity of the remainder partials
  static_assert(NTW >= 1 && KC >= 1 && 16 * KC <= 256, "shape");
  __shared__ __attribute__((aligned(16))) float lds[2 * SLOT + 2 * (RED > 0 ? RED : 4)];

  const int64_t M = eff_count(g.M, g.M_dev);
  const int64_t ntiles = cdiv(M, 16);
  const int64_t b0 = blockIdx.x, G = gridDim.x;
  if (b0 >= ntiles) return;
  const int64_t nmine = cdiv(ntiles - b0, G);
  const int64_t K = g.K, N = g.N;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int fr = lane & 15, fg = lane >> 4;
  const float* A = (const float*)g.A;
  const float* B = (const float*)g.B;
  const uint32_t base = (uint32_t)(uintptr_t)(lds_void_ptr)lds;
  const uint32_t red_base = base + 2u * SLOT * 4u;

  // DMA of one A tile: this wave's rows 4 wid .. 4 wid + 3, one instruction per
  // row, lane q < K/4 loading the row's 16-byte quad q.  Rows past M read row 0.
  const bool q_on = 4 * lane < K;
  const float* arow = A + (b0 * 16 + 4 * wid) * g.a_si + 4 * lane;   // row 4 wid of the block's current tile
  const int64_t a_step = G * 16 * g.a_si;
  auto issue = [&](int64_t tile, int slot) {
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      const int64_t gr = tile * 16 + 4 * wid + rr;
      const float* src = gr < M ? arow + rr * g.a_si : A + 4 * lane;
      if (q_on) dma::load16(src, base + (uint32_t)(slot * SLOT + (4 * wid + rr) * KS) * 4u);
    }
  };

  // zero the k tail of every row of both slots (never written by the DMA)
  for (int e = tid; e < 2 * 16 * (KS / 4); e += G_THREADS) {
    const int q = e % (KS / 4), row = e / (KS / 4);
    if (4 * q >= K) dma::ds_zero4(base + (uint32_t)(row * KS + 4 * q) * 4u);
  }
  issue(b0, 0);

  // B in registers (zero past K and N), then the bias of the register tiles
  float bw[NTW][KC][4];
  float br[NR > 0 ? NR : 1][KQ][4];
  auto bval = [&](int64_t k, int64_t j) -> float {
    return (k < K && j < N) ? B[k * g.b_sk + j * g.b_sj] : 0.f;
  };
#pragma unroll
  for (int t = 0; t < NTW; ++t) {
    const int64_t j = (int64_t)(wid * NTW + t) * 16 + fr;
#pragma unroll
    for (int c = 0; c < KC; ++c) {
      const int64_t k = 16 * c + 4 * fg;
      if (g.b_vec && k + 3 < K && j < N) {   // b_vec: B contiguous along k and 16-byte aligned
        const float4 v = *reinterpret_cast<const float4*>(B + j * g.b_sj + k);
        bw[t][c][0] = v.x; bw[t][c][1] = v.y; bw[t][c][2] = v.z; bw[t][c][3] = v.w;
      } else {
#pragma unroll
        for (int s = 0; s < 4; ++s) bw[t][c][s] = bval(k + s, j);
      }
    }
  }
#pragma unroll
  for (int q = 0; q < NR; ++q) {
    const int64_t j = (int64_t)(4 * NTW + q) * 16 + fr;
#pragma unroll
    for (int cc = 0; cc < KQ; ++cc) {
      const int c = 4 * cc + wid;
#pragma unroll
      for (int s = 0; s < 4; ++s) br[q][cc][s] = c < KC ? bval(16 * c + 4 * fg + s, j) : 0.f;
    }
  }
  float bias_w[NTW], bias_r[NR > 0 ? NR : 1];
#pragma unroll
  for (int t = 0; t < NTW; ++t) {
    const int64_t j = (int64_t)(wid * NTW + t) * 16 + fr;
    bias_w[t] = (g.bias && j < N) ? g.bias[j] : 0.f;
  }
#pragma unroll
  for (int q = 0; q < NR; ++q) {
    const int64_t j = (int64_t)(4 * NTW + q) * 16 + fr;
    bias_r[q] = (g.bias && j < N) ? g.bias[j] : 0.f;
  }

  // output columns of this lane: register tiles, then remainder tiles
  float* C = g.C;
  int64_t jw[NTW];
#pragma unroll
  for (int t = 0; t < NTW; ++t) jw[t] = (int64_t)(wid * NTW + t) * 16 + fr;
  // stores of one 16-row tile's register results (rows row0 + 4 fg + r)
  auto store_reg = [&](int64_t row0, int t, int r, float v) {
    const int64_t i = row0 + 4 * fg + r;
    if (i < M && jw[t] < N) C[i * g.ldc + jw[t]] = v + bias_w[t];
  };
  auto store_rem = [&](int64_t row0, int q, const f32x4& v) {
    const int64_t j = (int64_t)(4 * NTW + q) * 16 + fr;
    if (j >= N) return;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t i = row0 + 4 * fg + r;
      if (i < M) C[i * g.ldc + j] = v[r] + bias_r[q];
    }
  };
  auto read_partials = [&](int q, int par, f32x4 (&p)[4]) {
#pragma unroll
    for (int w = 0; w < 4; ++w)
      p[w] = dma::ds_read4(red_base + (uint32_t)(par * RED + ((q * 4 + w) * 64 + lane) * 4) * 4u);
  };

  const uint32_t a_lane = (uint32_t)(fr * KS + 4 * fg) * 4u;
  // One tile.  The previous tile's results (st_w, and the remainder partials in
  // LDS for the wave whose turn it is) are stored from inside this tile's chunk
  // loop, between MFMA groups, so the stores overlap the matrix work; they are
  // issued before the next tile's vmcnt(0), a whole tile later.
  auto body = [&](int64_t it, f32x4 (&st_w)[NTW], f32x4 (&cu_w)[NTW], f32x4 (&cu_r)[NR > 0 ? NR : 1]) {
    const int64_t tile = b0 + it * G;
    const int slot = (int)(it & 1);
    dma::wait_vm<0>();
    dma::wait_lgkm0();
    dma::barrier();   // tile `it` is in LDS; every wave is done with tile it - 1 (its slot, its partials are in LDS)
    const uint32_t a_base = base + (uint32_t)(slot * SLOT) * 4u + a_lane;
    f32x4 af[KC];
    af[0] = dma::ds_read4(a_base);
    if (it + 1 < nmine) {
      arow += a_step;
      issue(tile + G, slot ^ 1);
    }
    const bool prev = it >= 1;
    const bool reducer = NR > 0 && prev && wid == (int)((it - 1) & 3);
    const int64_t prow0 = (tile - G) * 16;

#pragma unroll
    for (int t = 0; t < NTW; ++t) cu_w[t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int q = 0; q < NR; ++q) cu_r[q] = f32x4{0.f, 0.f, 0.f, 0.f};
    f32x4 rp[4];
#pragma unroll
    for (int c = 0; c < KC; ++c) {
      dma::wait_lgkm0();
      if (c + 1 < KC) af[c + 1] = dma::ds_read4(a_base + (uint32_t)(16 * (c + 1)) * 4u);
      // af[c] passes through an asm statement placed after the wait and after the next
      // chunk's read: its MFMAs cannot be hoisted above that read, so the read's latency
      // hides behind them (and the two fragments never share registers)
      dma::tie(af[c]);
#pragma unroll
      for (int s = 0; s < 4; ++s) {
#pragma unroll
        for (int t = 0; t < NTW; ++t)
          cu_w[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[c][s], bw[t][c][s], cu_w[t], 0, 0, 0);
        if (s == 1 && prev) {   // previous tile, register results: two rows of a tile per chunk, early in
                                // the tile so they complete before the next tile's vmcnt(0)
#pragma unroll
          for (int k = 2 * c; k < 4 * NTW && k < 2 * c + 2; ++k) store_reg(prow0, k / 4, k % 4, st_w[k / 4][k % 4]);
        }
      }
      if (NR > 0 && (c & 3) == wid) {
#pragma unroll
        for (int s = 0; s < 4; ++s)
#pragma unroll
          for (int q = 0; q < NR; ++q)
            cu_r[q] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[c][s], br[q][c / 4][s], cu_r[q], 0, 0, 0);
      }
      if (reducer) {   // previous tile, remainder q: partials read at chunk 2q, summed and stored at 2q + 1
#pragma unroll
        for (int q = 0; q < NR; ++q) {
          if (c == (2 * q) % KC) read_partials(q, slot ^ 1, rp);
          if (c == (2 * q + 1) % KC) {
#pragma unroll
            for (int w = 0; w < 4; ++w) dma::tie(rp[w]);
            store_rem(prow0, q, ((rp[0] + rp[1]) + rp[2]) + rp[3]);
          }
        }
      }
      __builtin_amdgcn_sched_barrier(0);   // the chunk's work stays above the next chunk's wait
    }
#pragma unroll
    for (int q = 0; q < NR; ++q)
      dma::ds_write4(red_base + (uint32_t)(slot * RED + ((q * 4 + wid) * 64 + lane) * 4) * 4u, cu_r[q]);
  };

  f32x4 acc0[NTW], acc1[NTW], accr[NR > 0 ? NR : 1];
  int64_t it = 0;
  for (; it + 1 < nmine; it += 2) {
    body(it, acc1, acc0, accr);
    body(it + 1, acc0, acc1, accr);
  }
  if (it < nmine) body(it, acc1, acc0, accr);
  // the last tile: its register results are in acc0 if nmine is odd, else acc1
  dma::wait_lgkm0();
  dma::barrier();
  const int64_t last = nmine - 1;
  const int64_t lrow0 = (b0 + last * G) * 16;
#pragma unroll
  for (int t = 0; t < NTW; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r) store_reg(lrow0, t, r, (nmine & 1) ? acc0[t][r] : acc1[t][r]);
  if (NR > 0 && wid == (int)(last & 3)) {
#pragma unroll
    for (int q = 0; q < NR; ++q) {
      f32x4 p[4];
      read_partials(q, (int)(last & 1), p);
      dma::wait_lgkm0();
#pragma unroll
      for (int w = 0; w < 4; ++w) dma::tie(p[w]);
      store_rem(lrow0, q, ((p[0] + p[1]) + p[2]) + p[3]);
    }
  }
}

// Host side (gemm_rs.hip).  gemm_rs_applicable: an instance matches the shape
// (13 column tiles, K in (192, 224]: the key/value projection of 100-wide
// heads) and the fp32 operands meet the kernel's requirements.  gemm_rs_launch
// launches it with one block per CU (at most one per 16-row tile).
bool gemm_rs_applicable(const GemmArgs& g);
mtgnn_status gemm_rs_launch(const GemmArgs& g, hipStream_t s);

}  // namespace mtgnn

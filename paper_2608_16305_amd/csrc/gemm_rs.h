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
//
// TB = uint16_t (bfloat16 weights): the products run on v_mfma_f32_16x16x16_bf16, one per tile and chunk,
// with the register share of B packed to bfloat16 pairs.  A's rows are the bfloat16 mode's neighbour-slot
// inputs, which their producer stores already rounded to bfloat16, so their high halves are exact.
template <class Site, int NCT, int KC, int OCC, typename TB = float>
__global__ __launch_bounds__(G_THREADS, OCC) void k_gemm_rs(GemmArgs g) {
  constexpr bool BF = std::is_same<TB, uint16_t>::value;
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
  const TB* B = (const TB*)g.B;
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

  // B in registers (zero past K and N), then the bias of the register tiles; float32 weights as floats,
  // bfloat16 weights packed four to a register pair (the MFMA operand).  No load sits under a per-lane
  // condition: such a load is compiled into a branch of its own that waits for it, one memory round trip
  // per load.  The host admits only 16 (KC - 1) < K <= 16 KC and 16 (NCT - 1) < N <= 16 NCT, so only chunk
  // KC - 1 reaches past K, and with NR > 0 every register tile lies left of column 16 (NCT - 1) < N: those
  // loads need no test at all.  The others read a clamped index, and their value is replaced by zero after
  // the group's loads have been issued (the empty asm keeps each such load unconditional).
  float bw[BF ? 1 : NTW][BF ? 1 : KC][4];
  float br[BF || NR == 0 ? 1 : NR][BF ? 1 : KQ][4];
  s16x4 bwp[BF ? NTW : 1][BF ? KC : 1];
  s16x4 brp[BF && NR > 0 ? NR : 1][BF ? KQ : 1];
  constexpr bool REG_J_IN = NR > 0;
  auto raw_at = [&](int64_t k, int64_t j) -> uint32_t {   // bits of B(k, j), indices clamped into B
    const int64_t i = (k < K ? k : K - 1) * g.b_sk + (j < N ? j : N - 1) * g.b_sj;
    if constexpr (BF) return reinterpret_cast<const uint16_t*>(B)[i];
    else return __float_as_uint(reinterpret_cast<const float*>(B)[i]);
  };
  auto live = [](uint32_t& v) { asm volatile("" : "+v"(v)); };
  if (!BF && g.b_vec) {   // B contiguous along k and 16-byte aligned; K % 4 == 0, so k < K holds the whole quad
#pragma unroll
    for (int t = 0; t < NTW; ++t) {
      const int64_t j = (int64_t)(wid * NTW + t) * 16 + fr;
      const float* col = (const float*)B + (REG_J_IN || j < N ? j : N - 1) * g.b_sj;
      f32x4 v[KC];
#pragma unroll
      for (int c = 0; c < KC; ++c) {
        const int64_t k = 16 * c + 4 * fg;
        v[c] = *reinterpret_cast<const f32x4*>(col + (c < KC - 1 || k < K ? k : K - 4));
      }
#pragma unroll
      for (int c = 0; c < KC; ++c)
        if (c == KC - 1 || !REG_J_IN) dma::tie(v[c]);
#pragma unroll
      for (int c = 0; c < KC; ++c) {
        const bool ok = (c < KC - 1 || 16 * c + 4 * fg < K) && (REG_J_IN || j < N);
#pragma unroll
        for (int s = 0; s < 4; ++s) bw[t][c][s] = ok ? v[c][s] : 0.f;
      }
    }
  } else {
#pragma unroll
    for (int t = 0; t < NTW; ++t) {
      const int64_t j = (int64_t)(wid * NTW + t) * 16 + fr;
      uint32_t raw[KC][4];
#pragma unroll
      for (int c = 0; c < KC; ++c)
#pragma unroll
        for (int s = 0; s < 4; ++s) raw[c][s] = raw_at(16 * c + 4 * fg + s, j);
#pragma unroll
      for (int c = 0; c < KC; ++c)
#pragma unroll
        for (int s = 0; s < 4; ++s)
          if (c == KC - 1 || !REG_J_IN) live(raw[c][s]);
#pragma unroll
      for (int c = 0; c < KC; ++c) {
        uint32_t v[4];
#pragma unroll
        for (int s = 0; s < 4; ++s)
          v[s] = (c < KC - 1 || 16 * c + 4 * fg + s < K) && (REG_J_IN || j < N) ? raw[c][s] : 0u;
        if constexpr (BF) bwp[t][c] = s16x4{(short)v[0], (short)v[1], (short)v[2], (short)v[3]};
        else
#pragma unroll
          for (int s = 0; s < 4; ++s) bw[t][c][s] = __uint_as_float(v[s]);
      }
    }
  }
#pragma unroll
  for (int q = 0; q < NR; ++q) {   // remainder tiles: this wave's chunks c = 4 cc + wid (a chunk past KC reads as zero)
    const int64_t j = (int64_t)(4 * NTW + q) * 16 + fr;
    uint32_t raw[KQ][4];
#pragma unroll
    for (int cc = 0; cc < KQ; ++cc)
#pragma unroll
      for (int s = 0; s < 4; ++s) raw[cc][s] = raw_at(16 * (4 * cc + wid) + 4 * fg + s, j);
#pragma unroll
    for (int cc = 0; cc < KQ; ++cc)
#pragma unroll
      for (int s = 0; s < 4; ++s) live(raw[cc][s]);
#pragma unroll
    for (int cc = 0; cc < KQ; ++cc) {
      const int c = 4 * cc + wid;
      uint32_t v[4];
#pragma unroll
      for (int s = 0; s < 4; ++s) v[s] = c < KC && 16 * c + 4 * fg + s < K && j < N ? raw[cc][s] : 0u;
      if constexpr (BF) brp[q][cc] = s16x4{(short)v[0], (short)v[1], (short)v[2], (short)v[3]};
      else
#pragma unroll
        for (int s = 0; s < 4; ++s) br[q][cc][s] = __uint_as_float(v[s]);
    }
  }
  float bias_w[NTW], bias_r[NR > 0 ? NR : 1];
  {
    float v[NTW + NR];
#pragma unroll
    for (int t = 0; t < NTW + NR; ++t) {   // tile t: register tile t, then remainder tile t - NTW
      const int64_t j = (int64_t)(t < NTW ? wid * NTW + t : 4 * NTW + t - NTW) * 16 + fr;
      v[t] = g.bias ? g.bias[j < N ? j : N - 1] : 0.f;
    }
#pragma unroll
    for (int t = 0; t < NTW + NR; ++t) asm volatile("" : "+v"(v[t]));
#pragma unroll
    for (int t = 0; t < NTW + NR; ++t) {
      const int64_t j = (int64_t)(t < NTW ? wid * NTW + t : 4 * NTW + t - NTW) * 16 + fr;
      (t < NTW ? bias_w[t] : bias_r[t - NTW]) = j < N ? v[t] : 0.f;
    }
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
      if constexpr (BF) {
        const s16x4 ap = bf16x4_exact(float4{af[c][0], af[c][1], af[c][2], af[c][3]});
#pragma unroll
        for (int t = 0; t < NTW; ++t)
          cu_w[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(ap, bwp[t][c], cu_w[t], 0, 0, 0);
        if (prev) {   // previous tile, register results: two rows of a tile per chunk
#pragma unroll
          for (int k = 2 * c; k < 4 * NTW && k < 2 * c + 2; ++k) store_reg(prow0, k / 4, k % 4, st_w[k / 4][k % 4]);
        }
        if (NR > 0 && (c & 3) == wid) {
#pragma unroll
          for (int q = 0; q < NR; ++q)
            cu_r[q] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(ap, brp[q][c / 4], cu_r[q], 0, 0, 0);
        }
      } else {
#pragma unroll
        for (int s = 0; s < 4; ++s) {
#pragma unroll
          for (int t = 0; t < NTW; ++t)
            cu_w[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[c][s], bw[t][c][s], cu_w[t], 0, 0, 0);
          if (s == 1 && prev) {   // previous tile, register results: two rows of a tile per chunk, early in
                                  // the tile so they complete before the next tile's vmcnt(0)
#pragma unroll
            for (int k = 2 * c; k < 4 * NTW && k < 2 * c + 2; ++k)
              store_reg(prow0, k / 4, k % 4, st_w[k / 4][k % 4]);
          }
        }
        if (NR > 0 && (c & 3) == wid) {
#pragma unroll
          for (int s = 0; s < 4; ++s)
#pragma unroll
            for (int q = 0; q < NR; ++q)
              cu_r[q] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[c][s], br[q][c / 4][s], cu_r[q], 0, 0, 0);
        }
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
mtgnn_status gemm_rs_launch(const GemmArgs& g, hipStream_t s, bool bf16_weights);

}  // namespace mtgnn

namespace mtgnn {

namespace rs {
constexpr int dw_stride(int nt) {   // smallest stride >= 16 nt floats that is 16 mod 32
  return (16 * nt) % 32 == 16 ? 16 * nt : 16 * nt + 16;
}
}  // namespace rs

// Output-stationary weight gradient over many rows:
//   part[block][i][j] = sum over the block's rows p of X[p][i] Y[p][j],   i < NI 16, j < NJ 16,
// with X = the output gradient (dy, row stride ldx, nx = N_out valid columns) and
// Y = the layer input (row stride ldy, ny valid columns) followed by an
// all-ones column at j = ny (the bias gradient).  Rows come in 16-row chunks;
// block b takes chunks b, b + gridDim.x, ...; a fixed-order reduction over the
// blocks' partials (k_splitk_reduce) gives dW and db.
//
// Each of the 4 waves accumulates a fixed set of 16 x 16 output tiles for the
// whole launch: tile rows I = 3 wid .. 3 wid + 2 (all NJ tile columns) and, in
// the last tile row I = 12, the tile columns J = wid, wid + 4, ...  (NI = 13).
// Per chunk both operands go to LDS by direct global-to-LDS loads DW_RS_SLOTS - 1
// chunks ahead; MFMA sub-step s of a chunk takes rows 4 s + l/16 (lane l), reading one
// float per operand fragment.  Rows past the row count are zero-filled.
constexpr int DW_RS_SLOTS = 2;   // 2 or 3 (3, two chunks in flight, measured slower: 88 vs 85 us)

template <class Site, int NJ>
__global__ __launch_bounds__(G_THREADS, 1) void k_dw_rs(const float* __restrict__ X, int64_t ldx, int nx,
                                                     const float* __restrict__ Y, int64_t ldy, int ny, int64_t R,
                                                     const int32_t* R_dev, float* __restrict__ part) {
  constexpr int NI = 13, RW = 3;                 // tile rows: 3 per wave + the shared last one
  constexpr int EX = (NJ + 3) / 4;               // tiles of the last tile row per wave, at most
  constexpr int SX = rs::dw_stride(NI), SY = rs::dw_stride(NJ);
  constexpr int SLOT = 16 * (SX + SY);           // floats per chunk slot
  constexpr int NSL = DW_RS_SLOTS;               // chunk slots: NSL - 1 chunks in flight
  __shared__ __attribute__((aligned(16))) float lds[NSL * SLOT];

  const int64_t rows = eff_count(R, R_dev);
  const int64_t nchunks = cdiv(rows, 16);
  const int64_t b0 = blockIdx.x, G = gridDim.x;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int fr = lane & 15, fg = lane >> 4;
  const uint32_t base = (uint32_t)(uintptr_t)(lds_void_ptr)lds;

  // DMA of one chunk: this wave's rows 4 wid .. 4 wid + 3 of X and of Y; rows past
  // the row count are zero-filled instead
  auto issue = [&](int64_t chunk, int slot) {
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      const int r = 4 * wid + rr;
      const int64_t gr = chunk * 16 + r;
      const uint32_t dx = base + (uint32_t)(slot * SLOT + r * SX) * 4u;
      const uint32_t dy = base + (uint32_t)(slot * SLOT + 16 * SX + r * SY) * 4u;
      if (gr < rows) {
        if (4 * lane < nx) dma::load16(X + gr * ldx + 4 * lane, dx);
        if (4 * lane < ny) dma::load16(Y + gr * ldy + 4 * lane, dy);
      } else {
        if (4 * lane < nx) dma::ds_zero4(dx + 16u * lane);
        if (4 * lane < ny) dma::ds_zero4(dy + 16u * lane);
      }
    }
  };

  f32x4 acc[RW][NJ], acx[EX];
#pragma unroll
  for (int i = 0; i < RW; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int e = 0; e < EX; ++e) acx[e] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int64_t nmine = b0 < nchunks ? cdiv(nchunks - b0, G) : 0;
#pragma unroll
  for (int c = 0; c < NSL - 1; ++c)
    if (c < nmine) issue(b0 + c * G, c);
  // padding columns of every slot, while the first chunks load (the loads fill columns < nx, < ny):
  // X columns nx .. 16 NI and Y columns ny .. 16 NJ are zero except Y column ny, the all-ones column
  {
    const int cx = 16 * NI - nx, cw = cx + 16 * NJ - ny;
    for (int e = tid; e < NSL * 16 * cw; e += G_THREADS) {
      const int slot = e / (16 * cw), rem = e % (16 * cw), r = rem / cw, c = rem % cw;
      const uint32_t off = c < cx ? (uint32_t)(slot * SLOT + r * SX + nx + c)
                                  : (uint32_t)(slot * SLOT + 16 * SX + r * SY + ny + (c - cx));
      const float v = c == cx ? 1.f : 0.f;
      asm volatile("ds_write_b32 %0, %1" ::"v"(base + off * 4u), "v"(v) : "memory");
    }
  }
  // fragment addresses within a slot: X column 16 I + fr, Y column 16 J + fr, row 4 s + fg
  const uint32_t xa = (uint32_t)(fg * SX + 16 * RW * wid + fr) * 4u;
  const uint32_t xl = (uint32_t)(fg * SX + 16 * (NI - 1) + fr) * 4u;
  const uint32_t ya = (uint32_t)(16 * SX + fg * SY + fr) * 4u;
  auto read1 = [&](uint32_t addr) {
    float v;
    asm volatile("ds_read_b32 %0, %1" : "=v"(v) : "v"(addr));
    return v;
  };
  for (int64_t it = 0; it < nmine; ++it) {
    const int slot = (int)(it % NSL);
    // chunk `it` has landed once at most the later chunks' loads are outstanding: a full chunk is 8
    // loads per wave (4 rows of X and of Y); a partial one (only the last can be) is waited out too
    if (NSL == 3 && it + 1 < nmine && (b0 + (it + 1) * G + 1) * 16 <= rows)
      dma::wait_vm<8>();
    else
      dma::wait_vm<0>();
    dma::wait_lgkm0();
    dma::barrier();   // chunk `it` is in LDS; every wave is done with chunk it - 1's slot
    if (it + NSL - 1 < nmine) issue(b0 + (it + NSL - 1) * G, (int)((it + NSL - 1) % NSL));
    const uint32_t sb = base + (uint32_t)(slot * SLOT) * 4u;
    // fragments of sub-step s (rows 4 s + fg of the chunk); those of s + 1 are read while
    // the MFMAs of s run (they pass through asm statements after the next reads)
    float fx[4][RW + 1], fy[4][NJ], fe[4][EX];
    auto read_frags = [&](int s) {
      const uint32_t rx = sb + (uint32_t)(4 * s * SX) * 4u, ry = sb + (uint32_t)(4 * s * SY) * 4u;
#pragma unroll
      for (int i = 0; i < RW; ++i) fx[s][i] = read1(rx + xa + 64u * i);
      fx[s][RW] = read1(rx + xl);
#pragma unroll
      for (int j = 0; j < NJ; ++j) fy[s][j] = read1(ry + ya + 64u * j);
#pragma unroll
      for (int e = 0; e < EX; ++e) {   // branch-free: a tile past the last column reads the last one (never stored)
        const int J = wid + 4 * e < NJ ? wid + 4 * e : NJ - 1;
        fe[s][e] = read1(ry + ya + 64u * (uint32_t)J);
      }
    };
    read_frags(0);
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      dma::wait_lgkm0();
      if (s + 1 < 4) read_frags(s + 1);
#pragma unroll
      for (int i = 0; i <= RW; ++i) asm volatile("" : "+v"(fx[s][i]));
#pragma unroll
      for (int j = 0; j < NJ; ++j) asm volatile("" : "+v"(fy[s][j]));
#pragma unroll
      for (int e = 0; e < EX; ++e) asm volatile("" : "+v"(fe[s][e]));
#pragma unroll
      for (int i = 0; i < RW; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(fx[s][i], fy[s][j], acc[i][j], 0, 0, 0);
#pragma unroll
      for (int e = 0; e < EX; ++e)
        acx[e] = __builtin_amdgcn_mfma_f32_16x16x4f32(fx[s][RW], fe[s][e], acx[e], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);   // the sub-step's MFMAs stay above the next wait
    }
  }

  // this block's partial: [NI 16 (rows < nx)][ny + 1 columns]
  const int64_t ldp = ny + 1;
  float* out = part + b0 * (int64_t)nx * ldp;
  auto store = [&](int I, int J, const f32x4& v) {
    const int col = 16 * J + fr;
    if (col > ny) return;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = 16 * I + 4 * fg + r;
      if (row < nx) out[(int64_t)row * ldp + col] = v[r];
    }
  };
#pragma unroll
  for (int i = 0; i < RW; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j) store(RW * wid + i, j, acc[i][j]);
#pragma unroll
  for (int e = 0; e < EX; ++e)
    if (wid + 4 * e < NJ) store(NI - 1, wid + 4 * e, acx[e]);
}

// Batched output-stationary weight gradients for small outputs (nx <= 16 NI, ny + 1 <= 16 NJ),
// the chunk layout of k_dw_rs: each wave owns the tile columns J = wid, wid + 4, ... over all NI
// tile rows (a column past the last one is computed on a clamped copy and not stored).
// DW_OS_SLOTS LDS slots keep DW_OS_SLOTS - 1 chunks in flight.  Every full chunk is 8 DMA
// instructions per wave (4 rows of X and of Y), so the wait for the oldest one is vmcnt(8 n)
// with n full chunks issued after it; a partial chunk (the stream's last) is waited for with
// the chunks before it.
constexpr int DW_OS_SLOTS = 2;

template <int N>
__device__ __forceinline__ void wait_vm_chunks(int n) {   // vmcnt(8 n'), n' = min(n, N) (wave-uniform n)
  if constexpr (N > 0) {
    if (n >= N) {
      dma::wait_vm<8 * N>();
      return;
    }
    wait_vm_chunks<N - 1>(n);
  } else {
    dma::wait_vm<0>();
  }
}

template <int NI, int NJ>
__device__ __forceinline__ void dw_os_body(const DwOsProblem& q, int64_t rows, int64_t bi, float* lds) {
  constexpr int EJ = (NJ + 3) / 4;
  constexpr int SX = rs::dw_stride(NI), SY = rs::dw_stride(NJ);
  constexpr int SLOT = 16 * (SX + SY);
  const int nx = q.nx, ny = q.ny;
  const int64_t nchunks = cdiv(rows, 16), G = q.nblk;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int fr = lane & 15, fg = lane >> 4;
  const uint32_t base = (uint32_t)(uintptr_t)(lds_void_ptr)lds;
  const float* X = q.X;
  const float* Y = q.Y;

  auto issue = [&](int64_t chunk, int slot) {
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      const int r = 4 * wid + rr;
      const int64_t gr = chunk * 16 + r;
      const uint32_t dx = base + (uint32_t)(slot * SLOT + r * SX) * 4u;
      const uint32_t dy = base + (uint32_t)(slot * SLOT + 16 * SX + r * SY) * 4u;
      if (gr < rows) {
        if (4 * lane < nx) dma::load16(X + gr * q.ldx + 4 * lane, dx);
        if (4 * lane < ny) dma::load16(Y + gr * q.ldy + 4 * lane, dy);
      } else {
        if (4 * lane < nx) dma::ds_zero4(dx + 16u * lane);
        if (4 * lane < ny) dma::ds_zero4(dy + 16u * lane);
      }
    }
  };

  f32x4 acc[NI][EJ];
#pragma unroll
  for (int i = 0; i < NI; ++i)
#pragma unroll
    for (int e = 0; e < EJ; ++e) acc[i][e] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int64_t nmine = bi < nchunks ? cdiv(nchunks - bi, G) : 0;
  for (int c = 0; c < DW_OS_SLOTS - 1 && c < nmine; ++c) issue(bi + c * G, c);
  // padding columns of every slot, while the first chunks load (the loads fill columns < nx, < ny):
  // X columns nx .. 16 NI and Y columns ny .. 16 NJ are zero except Y column ny, the all-ones column
  {
    const int cx = 16 * NI - nx, cw = cx + 16 * NJ - ny;
    for (int e = tid; e < DW_OS_SLOTS * 16 * cw; e += G_THREADS) {
      const int slot = e / (16 * cw), rem = e % (16 * cw), r = rem / cw, c = rem % cw;
      const uint32_t off = c < cx ? (uint32_t)(slot * SLOT + r * SX + nx + c)
                                  : (uint32_t)(slot * SLOT + 16 * SX + r * SY + ny + (c - cx));
      const float v = c == cx ? 1.f : 0.f;
      asm volatile("ds_write_b32 %0, %1" ::"v"(base + off * 4u), "v"(v) : "memory");
    }
  }
  const uint32_t xa = (uint32_t)(fg * SX + fr) * 4u;
  const uint32_t ya = (uint32_t)(16 * SX + fg * SY + fr) * 4u;
  uint32_t yoff[EJ];
#pragma unroll
  for (int e = 0; e < EJ; ++e) {   // branch-free: a tile past the last column reads the last one
    const int J = wid + 4 * e < NJ ? wid + 4 * e : NJ - 1;
    yoff[e] = ya + 64u * (uint32_t)J;
  }
  auto read1 = [&](uint32_t addr) {
    float v;
    asm volatile("ds_read_b32 %0, %1" : "=v"(v) : "v"(addr));
    return v;
  };
  for (int64_t it = 0; it < nmine; ++it) {
    const int slot = (int)(it % DW_OS_SLOTS);
    // chunks issued after `it`: it + 1 .. last; the stream's partial last chunk counts as not full
    const int64_t last = it + DW_OS_SLOTS - 2 < nmine - 1 ? it + DW_OS_SLOTS - 2 : nmine - 1;
    const int after = (int)(last - it) - ((bi + last * G + 1) * 16 > rows && last > it ? 1 : 0);
    wait_vm_chunks<DW_OS_SLOTS - 2>(after);
    dma::wait_lgkm0();
    dma::barrier();   // chunk `it` is in LDS; every wave is done with chunk it - 1's slot
    if (it + DW_OS_SLOTS - 1 < nmine)
      issue(bi + (it + DW_OS_SLOTS - 1) * G, (int)((it + DW_OS_SLOTS - 1) % DW_OS_SLOTS));
    const uint32_t sb = base + (uint32_t)(slot * SLOT) * 4u;
    float fx[4][NI], fy[4][EJ];
    auto read_frags = [&](int s) {
      const uint32_t rx = sb + (uint32_t)(4 * s * SX) * 4u, ry = sb + (uint32_t)(4 * s * SY) * 4u;
#pragma unroll
      for (int i = 0; i < NI; ++i) fx[s][i] = read1(rx + xa + 64u * i);
#pragma unroll
      for (int e = 0; e < EJ; ++e) fy[s][e] = read1(ry + yoff[e]);
    };
    read_frags(0);
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      dma::wait_lgkm0();
      if (s + 1 < 4) read_frags(s + 1);
#pragma unroll
      for (int i = 0; i < NI; ++i) asm volatile("" : "+v"(fx[s][i]));
#pragma unroll
      for (int e = 0; e < EJ; ++e) asm volatile("" : "+v"(fy[s][e]));
#pragma unroll
      for (int i = 0; i < NI; ++i)
#pragma unroll
        for (int e = 0; e < EJ; ++e)
          acc[i][e] = __builtin_amdgcn_mfma_f32_16x16x4f32(fx[s][i], fy[s][e], acc[i][e], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  const int64_t ldp = ny + 1;
  float* out = q.part + bi * (int64_t)nx * ldp;
#pragma unroll
  for (int e = 0; e < EJ; ++e) {
    const int col = 16 * (wid + 4 * e) + fr;
    if (wid + 4 * e >= NJ || col > ny) continue;
#pragma unroll
    for (int i = 0; i < NI; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = 16 * i + 4 * fg + r;
        if (row < nx) out[(int64_t)row * ldp + col] = acc[i][e][r];
      }
  }
}

// One launch for the whole batch: block b works for the problem whose block range holds b.
template <class Site>   // the call site names the kernel symbol only
__global__ __launch_bounds__(G_THREADS, 1) void k_dw_os(DwOsBatch b) {
  constexpr int SLOT_MAX = 16 * (rs::dw_stride(7) + rs::dw_stride(13));
  __shared__ __attribute__((aligned(16))) float lds[DW_OS_SLOTS * SLOT_MAX];
  const int bx = blockIdx.x;
  int pi = 0;   // the problems' block ranges ascend
#pragma unroll
  for (int k = 1; k < DW_OS_MAXP; ++k)
    if (k < b.n && bx >= b.p[k].b_begin) pi = k;
  DwOsProblem q = b.p[pi];
  int64_t rows = eff_count(b.R, b.R_dev);
  if (q.row_den > 0) {   // only this row range can be nonzero: the rows are taken from its start
    const int64_t lo = rows * q.row_lo / q.row_den, hi = rows * q.row_hi / q.row_den;
    q.X += lo * q.ldx;
    q.Y += lo * q.ldy;
    rows = hi > lo ? hi - lo : 0;
  }
  if (q.ny + 1 <= 16 * 7) dw_os_body<7, 7>(q, rows, bx - q.b_begin, lds);
  else dw_os_body<7, 13>(q, rows, bx - q.b_begin, lds);
}

// Host side (gemm_rs.hip): dW[nx, ny] = X^T Y and db[nx] = column sums of X over R rows
// (clamped by R_dev), for nx in (192, 208] and ny + 1 <= 16 NJ with NJ in {13, 14}.
// part: workspace of dw_rs_ws_bytes(nx, ny).
bool dw_rs_applicable(const float* X, int64_t ldx, int nx, const void* Y, int y_dtype, int64_t ldy, int ny);
size_t dw_rs_ws_bytes(int nx, int ny);
mtgnn_status dw_rs_launch(const float* X, int64_t ldx, int nx, const float* Y, int64_t ldy, int ny, int64_t R,
                          const int32_t* R_dev, float* dW, int64_t lddw, float* db, void* ws, size_t ws_bytes,
                          hipStream_t s);

}  // namespace mtgnn

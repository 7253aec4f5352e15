// Device-wide primitives used by the step kernels: stable LSD radix sort of
// (key, value) pairs, exclusive scan of int32 counts, and deterministic column
// sums.  All are fixed-order, so their results do not depend on scheduling.
#include "common.h"

namespace mtgnn {

namespace {

constexpr int SORT_THREADS = 256;
constexpr int SORT_ITEMS = 4;
constexpr int SORT_TILE = SORT_THREADS * SORT_ITEMS;   // 1024 keys per block
constexpr int RADIX_BITS = 8;
constexpr int RADIX = 1 << RADIX_BITS;

constexpr int SCAN_THREADS = 256;
constexpr int SCAN_ITEMS = 16;
constexpr int SCAN_TILE = SCAN_THREADS * SCAN_ITEMS;
constexpr int SCAN1_THREADS = 1024;
constexpr int SCAN1_ITEMS = 32;
constexpr int64_t SCAN1_MAX = SCAN1_THREADS * SCAN1_ITEMS;   // one-block scan up to 32768 elements

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// ---------------------------------------------------------------- block scan helpers

// Exclusive scan of one int per thread across a 256-thread block; returns the block total.
__device__ int block_exclusive_scan(int v, int* out_excl, int* lds /* >= 4 ints */) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  int inc = v;
  for (int o = 1; o < 64; o <<= 1) {
    int t = __shfl_up(inc, o, 64);
    if (lane >= o) inc += t;
  }
  if (lane == 63) lds[wid] = inc;
  __syncthreads();
  int wave_off = 0, total = 0;
  for (int w = 0; w < SCAN_THREADS / 64; ++w) {
    int s = lds[w];
    if (w < wid) wave_off += s;
    total += s;
  }
  *out_excl = wave_off + inc - v;
  __syncthreads();
  return total;
}

// ---------------------------------------------------------------- scan kernels

__global__ __launch_bounds__(SCAN_THREADS) void k_scan_reduce(const int32_t* __restrict__ in, int64_t n,
                                                              int32_t* __restrict__ block_sums) {
  __shared__ int lds[8];
  const int64_t base = (int64_t)blockIdx.x * SCAN_TILE;
  int v[SCAN_ITEMS];   // every item loaded up front (an index past n reads element n - 1 and counts 0)
#pragma unroll
  for (int i = 0; i < SCAN_ITEMS; ++i) {
    const int64_t idx = base + (int64_t)i * SCAN_THREADS + threadIdx.x;
    v[i] = in[idx < n ? idx : n - 1];
  }
  int s = 0;
#pragma unroll
  for (int i = 0; i < SCAN_ITEMS; ++i) {
    keep_live(v[i]);
    s += base + (int64_t)i * SCAN_THREADS + threadIdx.x < n ? v[i] : 0;
  }
  int excl;
  int tot = block_exclusive_scan(s, &excl, lds);
  if (threadIdx.x == 0) block_sums[blockIdx.x] = tot;
}

// Scans one tile per block, adding a per-block offset (if given).
__global__ __launch_bounds__(SCAN_THREADS) void k_scan_tile(const int32_t* __restrict__ in, int32_t* __restrict__ out,
                                                            int64_t n, const int32_t* __restrict__ block_off,
                                                            int32_t* __restrict__ total) {
  __shared__ int lds[8];
  const int64_t base = (int64_t)blockIdx.x * SCAN_TILE + (int64_t)threadIdx.x * SCAN_ITEMS;
  int v[SCAN_ITEMS];
  int s = 0;
  for (int i = 0; i < SCAN_ITEMS; ++i) {
    int64_t idx = base + i;
    v[i] = idx < n ? in[idx] : 0;
    s += v[i];
  }
  int excl;
  int tot = block_exclusive_scan(s, &excl, lds);
  int off = (block_off ? block_off[blockIdx.x] : 0) + excl;
  for (int i = 0; i < SCAN_ITEMS; ++i) {
    int64_t idx = base + i;
    if (idx < n) out[idx] = off;
    off += v[i];
  }
  if (total && threadIdx.x == 0 && blockIdx.x == gridDim.x - 1)
    *total = (block_off ? block_off[blockIdx.x] : 0) + tot;
}

// One block of 1024 threads scans up to SCAN1_MAX elements.  The input is
// loaded coalesced (element i = j * 1024 + t goes to thread t) into LDS, then
// thread t scans the contiguous chunk [32 t, 32 t + 32) from LDS; one padding
// word per 32 keeps both access patterns free of bank conflicts.  The
// offsets go back through LDS and out coalesced.
__device__ __forceinline__ int scan1_pad(int i) { return i + (i >> 5); }

// ITEMS per thread (8, 16 or 32): the launcher takes the smallest that covers n, so a short scan does
// not pay for the padding's LDS traffic.
template <int ITEMS>
__global__ __launch_bounds__(SCAN1_THREADS) void k_scan_one_block(const int32_t* __restrict__ in,
                                                                  int32_t* __restrict__ out, int64_t n,
                                                                  int32_t* __restrict__ total) {
  constexpr int CAP = SCAN1_THREADS * ITEMS;
  __shared__ int buf[CAP + CAP / 32];
  __shared__ int wsum[SCAN1_THREADS / 64];
  const int t = threadIdx.x, lane = t & 63, wid = t >> 6;
  {
    const int last = (int)n - 1;   // n <= SCAN1_MAX: 32-bit offsets from the uniform base
    int x[ITEMS];   // every item loaded up front (an index past n reads element n - 1 and stores 0)
#pragma unroll
    for (int j = 0; j < ITEMS; ++j) {
      const int i = j * SCAN1_THREADS + t;
      x[j] = in[i < last ? i : last];
    }
#pragma unroll
    for (int j = 0; j < ITEMS; ++j) {
      const int i = j * SCAN1_THREADS + t;
      keep_live(x[j]);
      buf[scan1_pad(i)] = i < n ? x[j] : 0;
    }
  }
  __syncthreads();
  int v[ITEMS];
  int s = 0;
#pragma unroll
  for (int j = 0; j < ITEMS; ++j) {
    v[j] = buf[scan1_pad(t * ITEMS + j)];
    s += v[j];
  }
  int inc = s;
  for (int o = 1; o < 64; o <<= 1) {
    const int u = __shfl_up(inc, o, 64);
    if (lane >= o) inc += u;
  }
  if (lane == 63) wsum[wid] = inc;
  __syncthreads();
  int run = 0, tot = 0;
  for (int w = 0; w < SCAN1_THREADS / 64; ++w) {
    const int x = wsum[w];
    if (w < wid) run += x;
    tot += x;
  }
  run += inc - s;
#pragma unroll
  for (int j = 0; j < ITEMS; ++j) {
    buf[scan1_pad(t * ITEMS + j)] = run;
    run += v[j];
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < ITEMS; ++j) {
    const int i = j * SCAN1_THREADS + t;
    if (i < n) out[i] = buf[scan1_pad(i)];
  }
  if (total && t == 0) *total = tot;
}

// ---------------------------------------------------------------- radix sort kernels

__global__ __launch_bounds__(SORT_THREADS) void k_radix_hist(const uint32_t* __restrict__ keys, int64_t n, int shift,
                                                             int digit_bits, int nblk, int32_t* __restrict__ counts) {
  const uint32_t dmask = (1u << digit_bits) - 1u;
  __shared__ int hist[4][RADIX];
  const int wid = threadIdx.x >> 6;
  for (int i = threadIdx.x; i < 4 * RADIX; i += SORT_THREADS) (&hist[0][0])[i] = 0;
  __syncthreads();
  const int64_t base = (int64_t)blockIdx.x * SORT_TILE;
  uint32_t kk[SORT_ITEMS];   // the tile's keys loaded up front (an index past n reads key n - 1, not counted)
#pragma unroll
  for (int i = 0; i < SORT_ITEMS; ++i) {
    const int64_t idx = base + (int64_t)i * SORT_THREADS + threadIdx.x;
    kk[i] = keys[idx < n ? idx : n - 1];
  }
#pragma unroll
  for (int i = 0; i < SORT_ITEMS; ++i) {
    const int64_t idx = base + (int64_t)i * SORT_THREADS + threadIdx.x;
    keep_live(kk[i]);
    if (idx < n) atomicAdd(&hist[wid][(kk[i] >> shift) & dmask], 1);
  }
  __syncthreads();
  for (int d = threadIdx.x; d < (1 << digit_bits); d += SORT_THREADS)
    counts[(int64_t)d * nblk + blockIdx.x] = hist[0][d] + hist[1][d] + hist[2][d] + hist[3][d];
}

// Stable scatter: an item's destination is its digit's global offset for this
// block plus the number of same-digit items before it in the tile.  Tile order
// is round-major (round i covers items i*256 .. i*256+255, wave by wave).
__global__ __launch_bounds__(SORT_THREADS) void k_radix_scatter(const uint32_t* __restrict__ keys_in,
                                                                const uint32_t* __restrict__ vals_in,
                                                                uint32_t* __restrict__ keys_out,
                                                                uint32_t* __restrict__ vals_out, int64_t n, int shift,
                                                                int digit_bits, int nblk,
                                                                const int32_t* __restrict__ offsets) {
  __shared__ int run[RADIX];
  __shared__ int wcnt[4][RADIX];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  for (int d = threadIdx.x; d < (1 << digit_bits); d += SORT_THREADS) run[d] = offsets[(int64_t)d * nblk + blockIdx.x];
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  const int64_t base = (int64_t)blockIdx.x * SORT_TILE;
  uint32_t kk[SORT_ITEMS], vv[SORT_ITEMS];   // the tile's items, loaded up front
#pragma unroll
  for (int i = 0; i < SORT_ITEMS; ++i) {
    const int64_t idx = base + (int64_t)i * SORT_THREADS + threadIdx.x;
    kk[i] = idx < n ? keys_in[idx] : 0u;
    vv[i] = idx < n ? vals_in[idx] : 0u;
  }
#pragma unroll
  for (int i = 0; i < SORT_ITEMS; ++i) {
    for (int j = threadIdx.x; j < 4 * RADIX; j += SORT_THREADS) (&wcnt[0][0])[j] = 0;
    __syncthreads();
    const int64_t idx = base + (int64_t)i * SORT_THREADS + threadIdx.x;
    const bool valid = idx < n;
    const uint32_t key = kk[i];
    const uint32_t val = vv[i];
    const int d = (int)((key >> shift) & ((1u << digit_bits) - 1u));
    uint64_t peers = __ballot(valid);
    for (int b = 0; b < digit_bits; ++b) {
      const bool bit = (d >> b) & 1;
      const uint64_t m = __ballot(bit);
      peers &= bit ? m : ~m;
    }
    const int rank_w = __popcll(peers & lt_mask);
    const bool leader = valid && ((peers & lt_mask) == 0);
    if (leader) wcnt[wid][d] = __popcll(peers);
    __syncthreads();
    if (valid) {
      int pos = run[d] + rank_w;
      for (int w = 0; w < wid; ++w) pos += wcnt[w][d];
      keys_out[pos] = key;
      vals_out[pos] = val;
    }
    __syncthreads();
    for (int dd = threadIdx.x; dd < RADIX; dd += SORT_THREADS)
      run[dd] += wcnt[0][dd] + wcnt[1][dd] + wcnt[2][dd] + wcnt[3][dd];
    __syncthreads();
  }
}

// ---------------------------------------------------------------- column sums

constexpr int CS_COLS = 64;
constexpr int CS_ROWGROUPS = 4;
constexpr int CS_ROWS_PER_CHUNK = 128;   // 32 rows per thread: short dependent chains, many blocks

__global__ __launch_bounds__(256) void k_colsum_partial(const float* __restrict__ X, int64_t ld, int64_t rows,
                                                        const int32_t* __restrict__ rows_dev, int cols,
                                                        float* __restrict__ partial) {
  __shared__ float red[CS_ROWGROUPS][CS_COLS];
  const int c = blockIdx.x * CS_COLS + (threadIdx.x & 63);
  const int rg = threadIdx.x >> 6;
  const int64_t nrows = eff_count(rows, rows_dev);
  const int64_t r0 = (int64_t)blockIdx.y * CS_ROWS_PER_CHUNK;
  const int64_t r1 = min(nrows, r0 + CS_ROWS_PER_CHUNK);
  float s = 0.f;
  if (c < cols)
    for (int64_t r = r0 + rg; r < r1; r += CS_ROWGROUPS) s += X[r * ld + c];
  red[rg][threadIdx.x & 63] = s;
  __syncthreads();
  if (rg == 0 && c < cols)
    partial[(int64_t)blockIdx.y * cols + c] = ((red[0][threadIdx.x] + red[1][threadIdx.x]) + red[2][threadIdx.x]) +
                                              red[3][threadIdx.x];
}

// A wave per column: lane l adds chunks l, l + 64, ... in order, then a fixed butterfly.
__global__ void k_colsum_final(const float* __restrict__ partial, int nchunks, int cols, float* __restrict__ out,
                               int accumulate) {
  const int c = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (c >= cols) return;
  float s = 0.f;
  for (int j = lane; j < nchunks; j += 64) s += partial[(int64_t)j * cols + c];
  s = wave_sum(s);
  if (lane == 0) out[c] = accumulate ? out[c] + s : s;
}

}  // namespace

// ---------------------------------------------------------------- host wrappers

int bits_for(int64_t max_value) {
  int b = 0;
  while (b < 63 && (int64_t(1) << b) <= max_value) ++b;
  return b < 1 ? 1 : b;
}

size_t scan_ws_bytes(int64_t n) {
  if (n <= SCAN1_MAX) return 0;
  int64_t nb = cdiv(n, SCAN_TILE);
  return align256(sizeof(int32_t) * nb) * 2 + scan_ws_bytes(nb);
}

mtgnn_status scan_exclusive(const int32_t* in, int32_t* out, int64_t n, int32_t* total, void* ws, size_t ws_bytes,
                            hipStream_t s) {
  if (n <= 0) return MTGNN_OK;
  if (ws_bytes < scan_ws_bytes(n)) return MTGNN_EWORKSPACE;
  if (n <= SCAN_TILE) {
    k_scan_tile<<<1, SCAN_THREADS, 0, s>>>(in, out, n, nullptr, total);
    MTGNN_CHECK_LAUNCH("scan_tile");
    return MTGNN_OK;
  }
  if (n <= SCAN1_MAX) {
    if (n <= SCAN1_THREADS * 8)
      k_scan_one_block<8><<<1, SCAN1_THREADS, 0, s>>>(in, out, n, total);
    else if (n <= SCAN1_THREADS * 16)
      k_scan_one_block<16><<<1, SCAN1_THREADS, 0, s>>>(in, out, n, total);
    else
      k_scan_one_block<SCAN1_ITEMS><<<1, SCAN1_THREADS, 0, s>>>(in, out, n, total);
    MTGNN_CHECK_LAUNCH("scan_one_block");
    return MTGNN_OK;
  }
  const int64_t nb = cdiv(n, SCAN_TILE);
  char* w = (char*)ws;
  int32_t* sums = (int32_t*)w;
  int32_t* offs = (int32_t*)(w + align256(sizeof(int32_t) * nb));
  char* rest = w + 2 * align256(sizeof(int32_t) * nb);
  k_scan_reduce<<<(unsigned)nb, SCAN_THREADS, 0, s>>>(in, n, sums);
  MTGNN_CHECK_LAUNCH("scan_reduce");
  MTGNN_TRY(scan_exclusive(sums, offs, nb, nullptr, rest, ws_bytes - 2 * align256(sizeof(int32_t) * nb), s));
  k_scan_tile<<<(unsigned)nb, SCAN_THREADS, 0, s>>>(in, out, n, offs, total);
  MTGNN_CHECK_LAUNCH("scan_tile");
  return MTGNN_OK;
}

size_t radix_sort_ws_bytes(int64_t n) {
  const int64_t nblk = cdiv(n < 1 ? 1 : n, SORT_TILE);
  const int64_t nc = nblk * RADIX;
  return 2 * align256(sizeof(uint32_t) * n) + 2 * align256(sizeof(int32_t) * nc) + scan_ws_bytes(nc);
}

size_t radix_sort_result_bytes(int64_t n) { return 2 * align256(sizeof(uint32_t) * n); }

int radix_passes(int bits) { return (bits + RADIX_BITS - 1) / RADIX_BITS; }

void radix_sort_output(uint32_t** keys_io, uint32_t** vals_io, int64_t n, int bits, void* ws) {
  // an odd number of passes leaves the pairs in the first two workspace arrays
  if (n <= 1 || radix_passes(bits) % 2 == 0) return;
  *keys_io = (uint32_t*)ws;
  *vals_io = (uint32_t*)((char*)ws + align256(sizeof(uint32_t) * n));
}

mtgnn_status radix_sort_pairs(uint32_t** keys_io, uint32_t** vals_io, int64_t n, int bits, void* ws, size_t ws_bytes,
                              hipStream_t s) {
  if (n <= 1) return MTGNN_OK;
  uint32_t* keys = *keys_io;
  uint32_t* vals = *vals_io;
  if (ws_bytes < radix_sort_ws_bytes(n)) return MTGNN_EWORKSPACE;
  const int64_t nblk = cdiv(n, SORT_TILE);
  const int64_t nc = nblk * RADIX;
  char* w = (char*)ws;
  uint32_t* k2 = (uint32_t*)w;
  w += align256(sizeof(uint32_t) * n);
  uint32_t* v2 = (uint32_t*)w;
  w += align256(sizeof(uint32_t) * n);
  int32_t* counts = (int32_t*)w;
  w += align256(sizeof(int32_t) * nc);
  int32_t* offsets = (int32_t*)w;
  w += align256(sizeof(int32_t) * nc);
  const size_t rest = ws_bytes - (size_t)(w - (char*)ws);
  uint32_t *ki = keys, *vi = vals, *ko = k2, *vo = v2;
  // passes of equal width (at most 8 bits each), so each pass scans (2^width) x blocks counts
  const int passes = radix_passes(bits);
  const int width = (bits + passes - 1) / passes;
  for (int shift = 0; shift < bits; shift += width) {
    const int dbits = (bits - shift) < width ? (bits - shift) : width;
    k_radix_hist<<<(unsigned)nblk, SORT_THREADS, 0, s>>>(ki, n, shift, dbits, (int)nblk, counts);
    MTGNN_CHECK_LAUNCH("radix_hist");
    MTGNN_TRY(scan_exclusive(counts, offsets, ((int64_t)1 << dbits) * nblk, nullptr, w, rest, s));
    k_radix_scatter<<<(unsigned)nblk, SORT_THREADS, 0, s>>>(ki, vi, ko, vo, n, shift, dbits, (int)nblk, offsets);
    MTGNN_CHECK_LAUNCH("radix_scatter");
    uint32_t* t;
    t = ki; ki = ko; ko = t;
    t = vi; vi = vo; vo = t;
  }
  *keys_io = ki;   // the buffer holding the sorted pairs (the inputs or the first two workspace arrays)
  *vals_io = vi;
  return MTGNN_OK;
}

size_t colsum_ws_bytes(int64_t rows, int cols) {
  const int64_t nch = cdiv(rows < 1 ? 1 : rows, CS_ROWS_PER_CHUNK);
  return align256(sizeof(float) * nch * cols);
}

mtgnn_status colsum(const float* X, int64_t ld, int64_t rows, const int32_t* rows_dev, int cols, float* out,
                    bool accumulate, void* ws, size_t ws_bytes, hipStream_t s) {
  if (cols <= 0) return MTGNN_OK;
  const int64_t nch = cdiv(rows < 1 ? 1 : rows, CS_ROWS_PER_CHUNK);
  if (ws_bytes < colsum_ws_bytes(rows, cols)) return MTGNN_EWORKSPACE;
  float* partial = (float*)ws;
  dim3 g((unsigned)cdiv(cols, CS_COLS), (unsigned)nch);
  k_colsum_partial<<<g, 256, 0, s>>>(X, ld, rows, rows_dev, cols, partial);
  MTGNN_CHECK_LAUNCH("colsum_partial");
  k_colsum_final<<<(unsigned)cdiv(cols, 4), 256, 0, s>>>(partial, (int)nch, cols, out, accumulate ? 1 : 0);
  MTGNN_CHECK_LAUNCH("colsum_final");
  return MTGNN_OK;
}

}  // namespace mtgnn

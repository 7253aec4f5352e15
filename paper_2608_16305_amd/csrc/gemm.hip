// Split-K reduction and launch-shape helpers of the strip GEMM.
#include "gemm.h"

namespace mtgnn {

namespace {

// 64 outputs per block; the 4 waves sum interleaved split slices, combined in a fixed order.
// The partials are [nsplit][rows][ldp] (ldp 0: cols); rows i < dup_rows are also written to dup / dup_col.
__device__ __forceinline__ void splitk_reduce_body(const float* __restrict__ part, int64_t split_stride, int nsplit,
                                                   int64_t rows, int64_t cols, float* __restrict__ out, int64_t ldo,
                                                   int64_t ones_col, float* __restrict__ col_out,
                                                   float* __restrict__ out_hi = nullptr,
                                                   float* __restrict__ col_out_hi = nullptr, int64_t row_split = 0,
                                                   int64_t ldp = 0, float* __restrict__ dup = nullptr,
                                                   int64_t lddup = 0, int64_t dup_rows = 0,
                                                   float* __restrict__ dup_col = nullptr) {
  __shared__ float red[4][64];
  const int64_t e = (int64_t)blockIdx.x * 64 + (threadIdx.x & 63);
  const int g = threadIdx.x >> 6;
  int64_t i = e / cols;
  const int64_t j = e % cols;
  const int64_t pe = ldp > 0 ? i * ldp + j : e;
  float s = 0.f;
  if (e < rows * cols) {
    int z = g;
    for (; z + 60 < nsplit; z += 64) {   // sixteen loads in flight, added as four passes of the loop below
      float a[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) a[u] = part[(int64_t)(z + 4 * u) * split_stride + pe];
#pragma unroll
      for (int q = 0; q < 4; ++q) s += ((a[4 * q] + a[4 * q + 1]) + a[4 * q + 2]) + a[4 * q + 3];
    }
    for (; z + 12 < nsplit; z += 16) {   // four loads in flight
      const float a0 = part[(int64_t)z * split_stride + pe], a1 = part[(int64_t)(z + 4) * split_stride + pe];
      const float a2 = part[(int64_t)(z + 8) * split_stride + pe], a3 = part[(int64_t)(z + 12) * split_stride + pe];
      s += ((a0 + a1) + a2) + a3;
    }
    for (; z < nsplit; z += 4) s += part[(int64_t)z * split_stride + pe];
  }
  red[g][threadIdx.x & 63] = s;
  __syncthreads();
  if (g != 0 || e >= rows * cols) return;
  const int l = threadIdx.x;
  s = ((red[0][l] + red[1][l]) + red[2][l]) + red[3][l];
  if (i < dup_rows) {
    if (j == ones_col) {
      if (dup_col) dup_col[i] = s;
    } else if (dup) {
      dup[i * lddup + j] = s;
    }
  }
  if (out_hi && i >= row_split) {   // rows from row_split on go to the second output pair
    i -= row_split;
    out = out_hi;
    col_out = col_out_hi;
  }
  if (j == ones_col) col_out[i] = s;
  else out[i * ldo + j] = s;
}

struct ReduceProblem {
  const float* part;
  int64_t split_stride;
  int nsplit;
  int64_t rows, cols;
  float* out;
  int64_t ldo;
  int64_t ones_col;
  float* col_out;
  int64_t ldp = 0;
  float* dup = nullptr;
  int64_t lddup = 0, dup_rows = 0;
  float* dup_col = nullptr;
};
struct ReduceBatch {
  ReduceProblem p[DW_OS_MAXP];
  int n;
};

// blockIdx.y selects the problem; blocks past its outputs return before the barrier.
__global__ __launch_bounds__(256) void k_splitk_reduce_batch(ReduceBatch b) {
  if ((int)blockIdx.y >= b.n) return;
  const ReduceProblem& q = b.p[blockIdx.y];
  if ((int64_t)blockIdx.x * 64 >= q.rows * q.cols) return;
  splitk_reduce_body(q.part, q.split_stride, q.nsplit, q.rows, q.cols, q.out, q.ldo, q.ones_col, q.col_out, nullptr,
                     nullptr, 0, q.ldp, q.dup, q.lddup, q.dup_rows, q.dup_col);
}

}  // namespace

__global__ __launch_bounds__(256) void k_splitk_reduce(const float* __restrict__ part, int64_t split_stride,
                                                       int nsplit, int64_t rows, int64_t cols, float* __restrict__ out,
                                                       int64_t ldo, int64_t ones_col, float* __restrict__ col_out) {
  splitk_reduce_body(part, split_stride, nsplit, rows, cols, out, ldo, ones_col, col_out);
}

__global__ __launch_bounds__(256) void k_splitk_reduce_rows2(const float* __restrict__ part, int64_t split_stride,
                                                             int nsplit, int64_t rows, int64_t cols,
                                                             float* __restrict__ out, float* __restrict__ out_hi,
                                                             int64_t ldo, int64_t ones_col, float* __restrict__ col_out,
                                                             float* __restrict__ col_out_hi, int64_t row_split) {
  splitk_reduce_body(part, split_stride, nsplit, rows, cols, out, ldo, ones_col, col_out, out_hi, col_out_hi,
                     row_split);
}

int gemm_strip_width(int64_t N) {
  const int64_t per = cdiv(N, cdiv(N, 128));   // equal strips of at most 128 columns
  return per <= 32 ? 32 : per <= 64 ? 64 : per <= 112 ? 112 : 128;
}

int gemm_wide_strip_width(int64_t N) {
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
  return blocks < 1024 ? 32 : full;
}

// Up to 16 K reduction rows: 64 x 32 tiles over 256-row chunks (each block one
// short reduction; the grid is tiles x chunks).  Larger reductions keep full
// strips and cut the rows into chunks of >= 256 so the grid has about 1536
// blocks at the host row maximum (device-side counts often leave fewer active).
DwPlan dw_plan(int64_t R, int64_t N, int64_t K) {
  DwPlan p;
  const int64_t r = R < 1 ? 1 : R;
  if (r <= 16384) {
    p.bn = 32;
    p.bk = G_BK;
    p.kchunk = 256;
  } else {
    p.bn = gemm_wide_strip_width(K);
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

DwPlan dw_plan_dev(DwPlan host, int64_t tiles) {
  if (host.ksplit <= 1) return host;
  const int64_t want = cdiv(DW_DEV_BLOCKS, tiles < 1 ? 1 : tiles);
  host.ksplit = (int)(want < 1 ? 1 : want > host.ksplit ? host.ksplit : want);
  host.ksplit_dev = host.ksplit;
  return host;
}

// ---------------------------------------------------------------- batched products

mtgnn_status linear_fwd_batch(const FwdProblem* ps, int n, int64_t M, const int32_t* M_dev, int x_dtype,
                              int w_dtype, hipStream_t s) {
  if (n < 1 || n > G_MAXBATCH) return MTGNN_EINVAL;
  if (M <= 0) return MTGNN_OK;
  int64_t nmax = 1;
  for (int i = 0; i < n; ++i) nmax = ps[i].N > nmax ? ps[i].N : nmax;
  const int bn = gemm_tile_width(M, nmax, 1);
  GemmArgs gs[G_MAXBATCH];
  for (int i = 0; i < n; ++i) {
    GemmArgs g{};
    g.M = M; g.N = ps[i].N; g.K = ps[i].K; g.M_dev = M_dev;
    g.A = ps[i].x; g.a_si = ps[i].ldx; g.a_sk = 1;
    g.B = ps[i].W; g.b_sk = 1; g.b_sj = ps[i].ldw;
    g.C = ps[i].y; g.ldc = ps[i].ldy; g.bias = ps[i].bias;
    g.kchunk = ps[i].K; g.c_split_stride = 0;
    g.tile_bn = bn;
    gs[i] = g;
  }
  return gemm_batch_launch<site::Generic, true, true>(gs, n, 1, x_dtype, w_dtype, s);
}

namespace {
// One plan for the batch, from its largest output (with room for a bias column).
DwPlan dw_batch_plan(int64_t R, const int64_t* N, const int64_t* K, int n) {
  int best = 0;
  for (int i = 1; i < n; ++i)
    if (N[i] * (K[i] + 1) > N[best] * (K[best] + 1)) best = i;
  return dw_plan(R, N[best], K[best] + 1);
}
}  // namespace

namespace {

// Output-stationary batch (k_dw_os): every output at most 112 x 208 with its bias column, both
// operands at least 4 wide (every DMA instruction of a chunk has an active lane: the waits count them).
bool dw_os_shapes_ok(const int64_t* N, const int64_t* K, int n) {
  for (int i = 0; i < n; ++i)
    if (N[i] < 4 || N[i] > 112 || N[i] % 4 != 0 || K[i] < 4 || K[i] % 4 != 0 || K[i] + 1 > 208) return false;
  return true;
}

// Blocks per problem out of `total`, in proportion to the MFMAs per chunk (7 x 2 or 7 x 4 tiles a wave) times
// the share of the rows the problem reads (row_den > 0: (row_hi - row_lo) / row_den, else all).
void dw_os_split(const int64_t* K, int n, int total, int* nblk, const DwProblem* ps = nullptr) {
  int w[G_MAXBATCH], sum = 0;
  for (int i = 0; i < n; ++i) {
    w[i] = (cdiv(K[i] + 1, 16) <= 7 ? 2 : 4) * 12;
    if (ps && ps[i].row_den > 0) w[i] = w[i] * (ps[i].row_hi - ps[i].row_lo) / ps[i].row_den;
    if (w[i] < 1) w[i] = 1;
    sum += w[i];
  }
  int used = 0;
  for (int i = 0; i < n; ++i) {
    nblk[i] = (int)((int64_t)total * w[i] / sum);
    if (nblk[i] < 1) nblk[i] = 1;
    used += nblk[i];
  }
  for (int i = 0; used > total && i < n; ++i)   // only when rounding up single blocks overshot
    while (nblk[i] > 1 && used > total) --nblk[i], --used;
}

size_t dw_os_ws(const int64_t* N, const int64_t* K, int n, int total) {   // any split of `total` blocks fits
  size_t per = 0;
  for (int i = 0; i < n; ++i) per = std::max(per, sizeof(float) * (size_t)N[i] * (K[i] + 1));
  return per * (size_t)total + 256 * (size_t)n;
}

}  // namespace

size_t linear_dw_batch_ws_bytes(int64_t R, const int64_t* N, const int64_t* K, int n) {
  const DwPlan p = dw_batch_plan(R, N, K, n);
  size_t b = 0;
  if (p.ksplit > 1)
    for (int i = 0; i < n; ++i) b += (sizeof(float) * (size_t)p.ksplit * N[i] * (K[i] + 1) + 255) & ~size_t(255);
  if (dw_os_shapes_ok(N, K, n)) b = std::max(b, dw_os_ws(N, K, n, DW_OS_MAX_BLOCKS));
  return b;
}

template <class Site>
mtgnn_status linear_dw_batch(const DwProblem* ps, int n, int64_t R, const int32_t* R_dev, int x_dtype, void* ws,
                             size_t ws_bytes, hipStream_t s) {
  if (n < 1 || n > G_MAXBATCH) return MTGNN_EINVAL;
  int64_t Ns[G_MAXBATCH], Ks[G_MAXBATCH];
  for (int i = 0; i < n; ++i) {
    Ns[i] = ps[i].N;
    Ks[i] = ps[i].K;
  }
  if (ws_bytes < linear_dw_batch_ws_bytes(R, Ns, Ks, n)) return MTGNN_EWORKSPACE;
  bool os = x_dtype == MTGNN_F32 && dw_os_shapes_ok(Ns, Ks, n) && dw_os_cu_count() > 0;
  for (int i = 0; i < n && os; ++i)
    os = ps[i].db != nullptr && vec_ok(ps[i].dy, ps[i].lddy, sizeof(float)) &&
         vec_ok(ps[i].x, ps[i].ldx, sizeof(float));
  if (os) {   // one block per CU, blocks split over the problems; fixed-order reduce of the partials
    const int total = std::min(dw_os_cu_count(), DW_OS_MAX_BLOCKS);
    int nblk[G_MAXBATCH];
    dw_os_split(Ks, n, total, nblk, ps);
    DwOsBatch b{};
    ReduceBatch rb{};
    b.n = rb.n = n;
    b.R = R < 0 ? 0 : R;
    b.R_dev = R_dev;
    char* w = (char*)ws;
    int64_t max_out = 1, begin = 0;
    for (int i = 0; i < n; ++i) {
      const DwProblem& q = ps[i];
      const int64_t per = q.N * (q.K + 1);
      b.p[i] = DwOsProblem{q.dy, q.lddy, (const float*)q.x, q.ldx, (float*)w, (int)q.N, (int)q.K, (int)begin,
                           nblk[i], q.row_lo, q.row_hi, q.row_den};
      rb.p[i] = ReduceProblem{(const float*)w, per, nblk[i], q.N, q.K + 1, q.dW, q.lddw, q.K, q.db};
      w += (sizeof(float) * (size_t)nblk[i] * per + 255) & ~size_t(255);
      begin += nblk[i];
      max_out = std::max(max_out, per);
    }
    MTGNN_TRY(dw_os_launch(b, (int)begin, s));
    k_splitk_reduce_batch<<<dim3((unsigned)cdiv(max_out, 64), (unsigned)n), 256, 0, s>>>(rb);
    MTGNN_CHECK_LAUNCH("splitk_reduce_batch");
    return MTGNN_OK;
  }
  DwPlan plan = dw_batch_plan(R, Ns, Ks, n);
  if (R_dev) {
    int64_t tiles = 0;
    for (int i = 0; i < n; ++i) tiles += cdiv(Ns[i], 64 * G_WM) * cdiv(ps[i].db ? Ks[i] + 1 : Ks[i], plan.bn);
    plan = dw_plan_dev(plan, tiles);
  }
  GemmArgs gs[G_MAXBATCH];
  ReduceBatch rb{};
  rb.n = n;
  char* w = (char*)ws;
  int64_t max_out = 1;
  for (int i = 0; i < n; ++i) {
    const DwProblem& q = ps[i];
    const int64_t Kc = q.db ? q.K + 1 : q.K;
    GemmArgs g{};
    g.M = q.N; g.N = Kc; g.K = R < 1 ? 1 : R; g.K_dev = R_dev;
    if (q.db) { g.ones_col = q.K; g.col_out = q.db; }
    g.A = q.dy; g.a_si = 1; g.a_sk = q.lddy;
    g.B = q.x; g.b_sk = q.ldx; g.b_sj = 1;
    g.kchunk = plan.kchunk;
    g.ksplit_dev = plan.ksplit_dev;
    g.tile_bn = plan.bn;
    g.tile_bk = plan.bk;
    if (plan.ksplit == 1) {
      g.C = q.dW; g.ldc = q.lddw; g.c_split_stride = 0;
    } else {
      g.C = (float*)w; g.ldc = Kc; g.c_split_stride = q.N * Kc;
      rb.p[i] = ReduceProblem{(const float*)w, q.N * Kc, plan.ksplit, q.N, Kc, q.dW, q.lddw, q.db ? q.K : -1, q.db};
      w += (sizeof(float) * (size_t)plan.ksplit * q.N * Kc + 255) & ~size_t(255);
      max_out = q.N * Kc > max_out ? q.N * Kc : max_out;
    }
    gs[i] = g;
  }
  MTGNN_TRY((gemm_batch_launch<Site, false, false>(gs, n, plan.ksplit, MTGNN_F32, x_dtype, s)));
  if (plan.ksplit > 1) {
    k_splitk_reduce_batch<<<dim3((unsigned)cdiv(max_out, 64), (unsigned)n), 256, 0, s>>>(rb);
    MTGNN_CHECK_LAUNCH("splitk_reduce_batch");
  }
  return MTGNN_OK;
}

// Blocks per tile: the launch's blocks (one per CU, at most DW_OS_MAX_BLOCKS) in proportion to each
// tile's MFMAs per row chunk (7 x 2 or 7 x 4 tiles a wave), at least one each.
static int dw_tiles_split(const DwTile* t, int n, int* nblk) {
  int64_t K[DW_OS_MAXP];
  for (int i = 0; i < n; ++i) K[i] = t[i].ny;
  const int total = std::max(std::min(dw_os_cu_count(), DW_OS_MAX_BLOCKS), n);
  int w[DW_OS_MAXP], sum = 0;
  for (int i = 0; i < n; ++i) sum += (w[i] = cdiv(K[i] + 1, 16) <= 7 ? 2 : 4);
  int used = 0;
  for (int i = 0; i < n; ++i) used += (nblk[i] = std::max(1, (int)((int64_t)total * w[i] / sum)));
  return used;
}

static bool dw_tiles_shapes_ok(const DwTile* t, int n) {
  if (n < 1 || n > DW_OS_MAXP) return false;
  for (int i = 0; i < n; ++i) {
    const DwTile& q = t[i];
    if (q.nx < 4 || q.nx > 112 || q.nx % 4 || q.ny < 4 || q.ny > 108 || q.ny % 4) return false;
  }
  return true;
}

static bool dw_tiles_ok(const DwTile* t, int n) {
  if (!dw_tiles_shapes_ok(t, n)) return false;
  for (int i = 0; i < n; ++i) {
    const DwTile& q = t[i];
    if (!vec_ok(q.X, q.ldx, 4) || !vec_ok(q.Y, q.ldy, 4) || (q.dup_rows > 0 && !q.dup && !q.dup_db)) return false;
  }
  return true;
}

size_t dw_tiles_ws_bytes(const DwTile* t, int n) {   // depends on the shapes only
  if (!dw_tiles_shapes_ok(t, n)) return 0;
  int nblk[DW_OS_MAXP];
  dw_tiles_split(t, n, nblk);
  size_t b = 0;
  for (int i = 0; i < n; ++i) b += (sizeof(float) * (size_t)nblk[i] * t[i].nx * (t[i].ny + 1) + 255) & ~size_t(255);
  return b;
}

template <class Site>
mtgnn_status dw_tiles(const DwTile* t, int n, int64_t R, const int32_t* R_dev, void* ws, size_t ws_bytes,
                      hipStream_t s) {
  if (!dw_tiles_ok(t, n) || dw_os_cu_count() <= 0) return MTGNN_EUNSUPPORTED;
  if (ws_bytes < dw_tiles_ws_bytes(t, n)) return MTGNN_EWORKSPACE;
  int nblk[DW_OS_MAXP];
  dw_tiles_split(t, n, nblk);
  DwOsBatch b{};
  ReduceBatch rb{};
  b.n = rb.n = n;
  b.R = R < 0 ? 0 : R;
  b.R_dev = R_dev;
  char* w = (char*)ws;
  int64_t max_out = 1;
  int begin = 0;
  for (int i = 0; i < n; ++i) {
    const DwTile& q = t[i];
    const int64_t per = (int64_t)q.nx * (q.ny + 1);
    b.p[i] = DwOsProblem{q.X, q.ldx, q.Y, q.ldy, (float*)w, q.nx, q.ny, begin, nblk[i]};
    ReduceProblem rp{(const float*)w, per, nblk[i], q.nx, q.db ? q.ny + 1 : q.ny, q.dW, q.lddw, q.db ? q.ny : -1,
                     q.db};
    rp.ldp = q.ny + 1;
    rp.dup = q.dup;
    rp.lddup = q.lddup;
    rp.dup_rows = q.dup_rows;
    rp.dup_col = q.dup_db;
    rb.p[i] = rp;
    w += (sizeof(float) * (size_t)nblk[i] * per + 255) & ~size_t(255);
    begin += nblk[i];
    max_out = std::max(max_out, per);
  }
  MTGNN_TRY(dw_os_launch<Site>(b, begin, s));
  k_splitk_reduce_batch<<<dim3((unsigned)cdiv(max_out, 64), (unsigned)n), 256, 0, s>>>(rb);
  MTGNN_CHECK_LAUNCH("splitk_reduce_batch");
  return MTGNN_OK;
}

template mtgnn_status dw_tiles<site::Generic>(const DwTile*, int, int64_t, const int32_t*, void*, size_t, hipStream_t);
template mtgnn_status dw_tiles<site::GruDw>(const DwTile*, int, int64_t, const int32_t*, void*, size_t, hipStream_t);

template mtgnn_status linear_dw_batch<site::Generic>(const DwProblem*, int, int64_t, const int32_t*, int, void*, size_t,
                                                     hipStream_t);
template mtgnn_status linear_dw_batch<site::GruDw>(const DwProblem*, int, int64_t, const int32_t*, int, void*, size_t,
                                                   hipStream_t);

size_t dw_rs_ws_bytes(int nx, int ny);

size_t linear_dw_ws_bytes(int64_t R, int64_t N, int64_t K) {
  const DwPlan p = dw_plan(R, N, K + 1);
  size_t b = p.ksplit > 1 ? sizeof(float) * (size_t)p.ksplit * N * (K + 1) : 0;
  const int64_t nj = cdiv(K + 1, 16);
  if (N > 192 && N <= 208 && (nj == 13 || nj == 14)) {   // shapes the output-stationary kernel may take
    const size_t r = dw_rs_ws_bytes((int)N, (int)K);
    b = r > b ? r : b;
  }
  return b;
}

}  // namespace mtgnn

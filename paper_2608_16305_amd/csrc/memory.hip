// Memory phase of the batch step: batch intake, most-recent aggregation,
// message construction, GRU update with write-back, and their backward passes.
#include "gemm.h"
#include "ops.h"

namespace mtgnn {

namespace {

size_t a256(size_t x) { return (x + 255) & ~size_t(255); }

// ---------------------------------------------------------------- batch intake

__global__ void k_set_int(int32_t* p, int32_t v) { *p = v; }

__global__ void k_queries_all(const int32_t* __restrict__ src, const int32_t* __restrict__ dst,
                              const int32_t* __restrict__ neg, const float* __restrict__ t, int64_t n,
                              int32_t* __restrict__ q_node, float* __restrict__ q_t, int32_t* __restrict__ n_q) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i == 0) *n_q = (int32_t)(3 * n);
  if (i >= n) return;
  const float ti = t[i];
  q_node[i] = src[i];
  q_node[n + i] = dst[i];
  q_node[2 * n + i] = neg[i];
  q_t[i] = ti;
  q_t[n + i] = ti;
  q_t[2 * n + i] = ti;
}

__global__ void k_target_flags(const uint8_t* __restrict__ flags, int64_t n, int32_t* __restrict__ tgt) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) tgt[i] = (flags[i] & 3) == 0 ? 1 : 0;
}

__global__ void k_queries_masked(const int32_t* __restrict__ src, const int32_t* __restrict__ dst,
                                 const int32_t* __restrict__ neg, const float* __restrict__ t,
                                 const uint8_t* __restrict__ flags, int64_t n, const int32_t* __restrict__ pos,
                                 const int32_t* __restrict__ n_tar, int32_t* __restrict__ q_node,
                                 float* __restrict__ q_t, int32_t* __restrict__ n_q) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t nt = *n_tar;
  if (i == 0) *n_q = (int32_t)(3 * nt);
  if (i >= n || (flags[i] & 3) != 0) return;
  const int64_t p = pos[i];
  const float ti = t[i];
  q_node[p] = src[i];
  q_node[nt + p] = dst[i];
  q_node[2 * nt + p] = neg[i];
  q_t[p] = ti;
  q_t[nt + p] = ti;
  q_t[2 * nt + p] = ti;
}

// ---------------------------------------------------------------- most-recent aggregation

// Message m = 2i + role goes to src[i] (role 0) or dst[i] (role 1); pruned
// events get the sentinel key n_nodes, which sorts after every node.
// Most-recent aggregation through a node-indexed table T in the workspace.
// Message m = 2i + role of a non-pruned event i goes to node(m) (src for role
// 0, dst for role 1).  Under the batch order precondition ((t, eid) ascending,
// unique eids) the message with the largest (t, eid, role) is the one with
// the largest index, so T[node] = max m over the node's messages.  The max is
// taken with integer atomics (its value does not depend on their order); the
// entries are first reset for exactly the nodes of this batch, so the table
// needs no initialisation.  The winners (m == T[node(m)]) are then compacted in
// increasing m.
__device__ __forceinline__ int32_t msg_node(const int32_t* src, const int32_t* dst, const uint8_t* flags, int64_t m) {
  const int64_t i = m >> 1;
  if (flags != nullptr && (flags[i] & 2)) return -1;   // pruned: no message
  return (m & 1) ? dst[i] : src[i];
}

__global__ void k_agg_reset(const int32_t* __restrict__ src, const int32_t* __restrict__ dst,
                            const uint8_t* __restrict__ flags, int64_t nm, int32_t* __restrict__ T) {
  const int64_t m = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (m >= nm) return;
  const int32_t node = msg_node(src, dst, flags, m);
  if (node >= 0) T[node] = -1;
}

// Messages of one wave are consecutive, so among the wave's messages to one node
// the largest index is the highest such lane: only that lane issues the atomic
// (hub nodes receive hundreds of messages per batch; this bounds their atomics
// by the number of waves).
__global__ void k_agg_max(const int32_t* __restrict__ src, const int32_t* __restrict__ dst,
                          const uint8_t* __restrict__ flags, int64_t nm, int32_t* __restrict__ T) {
  const int64_t m = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int lane = threadIdx.x & 63;
  const int32_t node = m < nm ? msg_node(src, dst, flags, m) : -1;
  uint64_t pending = __ballot(node >= 0);
  while (pending) {   // one pass per distinct node of the wave
    const int leader = __ffsll((unsigned long long)pending) - 1;
    const int32_t v = __builtin_amdgcn_readlane(node, leader);
    const uint64_t same = __ballot(node == v);
    if (lane == 63 - __clzll(same)) atomicMax(&T[v], (int32_t)m);
    pending &= ~same;
  }
}

constexpr int AGG_BLOCK_THREADS = 1024;
constexpr int AGG_PER_THREAD = 16;
constexpr int64_t AGG_BLOCK_MAX = AGG_BLOCK_THREADS * AGG_PER_THREAD;

// One block compacts up to AGG_BLOCK_MAX messages: thread t owns messages 16 t .. 16 t + 15 (so
// the output order, increasing m, is thread order), flags its winners (m == T[node(m)]), and
// one block-wide exclusive scan of the per-thread winner counts gives every winner its
// position.  Each thread's loads are issued together (clamped indices, no branches), so the
// block waits for two rounds of memory latency rather than one per message.
__global__ __launch_bounds__(AGG_BLOCK_THREADS) void k_agg_compact_block(const int32_t* __restrict__ src,
                                                                         const int32_t* __restrict__ dst,
                                                                         const uint8_t* __restrict__ flags,
                                                                         int64_t nm, const int32_t* __restrict__ T,
                                                                         int32_t* __restrict__ uniq,
                                                                         int32_t* __restrict__ winner,
                                                                         int32_t* __restrict__ n_uniq) {
  __shared__ int wsum[AGG_BLOCK_THREADS / 64];
  const int t = threadIdx.x, lane = t & 63, wid = t >> 6;
  const int64_t m0 = (int64_t)t * AGG_PER_THREAD;
  int32_t node[AGG_PER_THREAD];
  {   // messages 2 i, 2 i + 1 of events i = m0 / 2 ..
    const int64_t ne = nm >> 1, e0 = m0 >> 1;
    // without flags, bytes of src stand in for them (in bounds: src holds 4 ne bytes) under a zero mask
    const uint8_t* fl = flags != nullptr ? flags : (const uint8_t*)src;
    const uint8_t pruned = flags != nullptr ? 2 : 0;
#pragma unroll
    for (int k = 0; k < AGG_PER_THREAD / 2; ++k) {
      const int64_t i = e0 + k < ne ? e0 + k : ne - 1;
      const int32_t a = src[i], b = dst[i];
      const uint8_t f = fl[i];
      const bool ok = (e0 + k < ne) & ((f & pruned) == 0);
      node[2 * k] = ok ? a : -1;
      node[2 * k + 1] = ok ? b : -1;
    }
  }
  int32_t tv[AGG_PER_THREAD];   // entry 0 stands in for a missing message
#pragma unroll
  for (int j = 0; j < AGG_PER_THREAD; ++j) tv[j] = T[node[j] >= 0 ? node[j] : 0];
  uint32_t winbits = 0;
#pragma unroll
  for (int j = 0; j < AGG_PER_THREAD; ++j)
    winbits |= (node[j] >= 0 && tv[j] == (int32_t)(m0 + j)) ? 1u << j : 0u;
  const int cnt = __popc(winbits);
  int incl = cnt;   // inclusive scan over the wave
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int v = __shfl_up(incl, o, 64);
    if (lane >= o) incl += v;
  }
  if (lane == 63) wsum[wid] = incl;
  __syncthreads();
  int base = 0, total = 0;
#pragma unroll
  for (int w = 0; w < AGG_BLOCK_THREADS / 64; ++w) {
    const int c = wsum[w];
    base += w < wid ? c : 0;
    total += c;
  }
  int pos = base + incl - cnt;
#pragma unroll
  for (int j = 0; j < AGG_PER_THREAD; ++j) {
    if ((winbits >> j) & 1u) {
      uniq[pos] = node[j];
      winner[pos] = (int32_t)(m0 + j);
      ++pos;
    }
  }
  if (t == 0) *n_uniq = total;
}

__global__ void k_agg_flags(const int32_t* __restrict__ src, const int32_t* __restrict__ dst,
                            const uint8_t* __restrict__ flags, int64_t nm, const int32_t* __restrict__ T,
                            int32_t* __restrict__ win) {
  const int64_t m = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (m >= nm) return;
  const int32_t node = msg_node(src, dst, flags, m);
  win[m] = (node >= 0 && T[node] == (int32_t)m) ? 1 : 0;
}

__global__ void k_agg_write(const int32_t* __restrict__ src, const int32_t* __restrict__ dst,
                            const uint8_t* __restrict__ flags, int64_t nm, const int32_t* __restrict__ win,
                            const int32_t* __restrict__ pos, int32_t* __restrict__ uniq,
                            int32_t* __restrict__ winner) {
  const int64_t m = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (m >= nm || !win[m]) return;
  uniq[pos[m]] = msg_node(src, dst, flags, m);
  winner[pos[m]] = (int32_t)m;
}

// ---------------------------------------------------------------- message construction

// One wave per row; lanes stride over the message columns.
template <typename T>
__global__ __launch_bounds__(256) void k_build_messages(const int32_t* __restrict__ src, const int32_t* __restrict__ dst,
                                                        const int32_t* __restrict__ eid, const float* __restrict__ t,
                                                        const int32_t* __restrict__ uniq,
                                                        const int32_t* __restrict__ winner,
                                                        const int32_t* __restrict__ n_rows, int64_t max_rows,
                                                        const T* __restrict__ mem, const float* __restrict__ lu,
                                                        const float* __restrict__ x, const float* __restrict__ tw,
                                                        const float* __restrict__ tb, int dm, int dt_dim, int de,
                                                        T* __restrict__ msg, float* __restrict__ dt_out) {
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= eff_count(max_rows, n_rows)) return;
  const int32_t w = winner[r];
  const int64_t i = w >> 1;
  const int64_t node = uniq[r];
  const int64_t partner = (w & 1) ? src[i] : dst[i];
  const float dt = t[i] - lu[node];
  const int dmsg = 2 * dm + dt_dim + de;
  T* out = msg + r * dmsg;
  const T* mn = mem + node * dm;
  const T* mp = mem + partner * dm;
  for (int c = lane; c < dm; c += 64) {
    out[c] = mn[c];
    out[dm + c] = mp[c];
  }
  for (int j = lane; j < dt_dim; j += 64) {
    const float arg = time_arg(tw[j], dt, tb[j]);
    Elem<T>::store(out, 2 * dm + j, sizeof(T) == 2 ? cos_for_bf16(arg) : cosf(arg));
  }
  if (de > 0) {
    const float* xr = x + (int64_t)eid[i] * de;
    for (int c = lane; c < de; c += 64) Elem<T>::store(out, 2 * dm + dt_dim + c, xr[c]);
  }
  if (lane == 0) dt_out[r] = dt;
}

// ---------------------------------------------------------------- GRU

template <typename T>
__global__ void k_gather_rows(const T* __restrict__ mem, const int32_t* __restrict__ uniq,
                              const int32_t* __restrict__ n_rows, int64_t max_rows, int dm, float* __restrict__ out) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t r = e / dm;
  if (r >= eff_count(max_rows, n_rows)) return;
  const int c = (int)(e % dm);
  out[e] = Elem<T>::load(mem, (int64_t)uniq[r] * dm + c);
}

// G = [gi | gh] (row stride 6 dm).  Writes the new memory row, last_update and the saved gates.
// Optional side job (wt.dst set): the zero-padded W_ih[:, col0 : col0 + dt]^T for the backward's fused
// time-feature gradient, written by every thread before the row test (grid-stride).
struct GruWT {
  const float* W_ih;
  float* dst;
  int rows, cols, dt, K, ld, col0;
};

template <typename T>
__global__ void k_gru_gates(const float* __restrict__ G, const float* __restrict__ h_old, int64_t ldh,
                            const int32_t* __restrict__ uniq, const int32_t* __restrict__ winner,
                            const float* __restrict__ t, const int32_t* __restrict__ n_rows, int64_t max_rows, int dm,
                            T* __restrict__ mem, float* __restrict__ lu, float* __restrict__ sr, float* __restrict__ sz,
                            float* __restrict__ sn, float* __restrict__ sghn, GruWT wt) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (wt.dst)
    for (int64_t x = e; x < (int64_t)wt.rows * wt.cols; x += (int64_t)gridDim.x * blockDim.x) {
      const int rr = (int)(x / wt.cols), cc = (int)(x % wt.cols);
      wt.dst[x] = (rr < wt.dt && cc < wt.K) ? wt.W_ih[(int64_t)cc * wt.ld + wt.col0 + rr] : 0.f;
    }
  const int64_t r = e / dm;
  if (r >= eff_count(max_rows, n_rows)) return;
  const int j = (int)(e % dm);
  const float* g = G + r * 6 * dm;
  const float rr = sigmoidf_(g[j] + g[3 * dm + j]);
  const float zz = sigmoidf_(g[dm + j] + g[4 * dm + j]);
  const float ghn = g[5 * dm + j];
  const float nn = tanhf(g[2 * dm + j] + rr * ghn);
  const float h = h_old[r * ldh + j];
  const float hn = (1.f - zz) * nn + zz * h;
  const int64_t node = uniq[r];
  Elem<T>::store(mem, node * dm + j, hn);
  if (j == 0) lu[node] = t[winner[r] >> 1];
  if (sr) {
    sr[e] = rr;
    sz[e] = zz;
    sn[e] = nn;
    sghn[e] = ghn;
  }
}

__global__ void k_gru_bwd_gates(const float* __restrict__ dh, const float* __restrict__ h_old, int64_t ldh,
                                const float* __restrict__ sr, const float* __restrict__ sz,
                                const float* __restrict__ sn, const float* __restrict__ sghn,
                                const int32_t* __restrict__ n_rows, int64_t max_rows, int dm, float* __restrict__ dgi,
                                float* __restrict__ dgh) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t r = e / dm;
  if (r >= eff_count(max_rows, n_rows)) return;
  const int j = (int)(e % dm);
  const float d = dh[e], rr = sr[e], zz = sz[e], nn = sn[e], ghn = sghn[e], h = h_old[r * ldh + j];
  const float dn_pre = d * (1.f - zz) * (1.f - nn * nn);
  const float dz_pre = d * (h - nn) * zz * (1.f - zz);
  const float dr_pre = dn_pre * ghn * rr * (1.f - rr);
  float* gi = dgi + r * 3 * dm;
  float* gh = dgh + r * 3 * dm;
  gi[j] = dr_pre;
  gi[dm + j] = dz_pre;
  gi[2 * dm + j] = dn_pre;
  gh[j] = dr_pre;
  gh[dm + j] = dz_pre;
  gh[2 * dm + j] = dn_pre * rr;
}

// ---------------------------------------------------------------- time-encoder gradients

constexpr int TG_ROWS = 32;   // rows per partial (8 per wave)

// Elapsed time of each row: delta[r] (delta == nullptr: 0, the query-side phi(0)).
struct RowDelta {
  const float* delta;
  __device__ bool get(int64_t r, float& d) const {
    d = delta ? delta[r] : 0.f;
    return true;
  }
};

template <typename D>
__global__ __launch_bounds__(256) void k_timegrad_partial(const float* __restrict__ dphi, int64_t ld, int64_t rows,
                                                          const int32_t* __restrict__ rows_dev, D delta,
                                                          const float* __restrict__ tw, const float* __restrict__ tb,
                                                          const float* __restrict__ sin_saved, int dt_dim,
                                                          float* __restrict__ part) {
  __shared__ float red_w[4][64], red_b[4][64];
  const int j = blockIdx.x * 64 + (threadIdx.x & 63);
  const int rg = threadIdx.x >> 6;
  const int64_t nrows = eff_count(rows, rows_dev);
  const int64_t r0 = (int64_t)blockIdx.y * TG_ROWS;
  const int64_t r1 = min(nrows, r0 + TG_ROWS);
  float sw = 0.f, sb = 0.f;
  if (j < dt_dim) {
    const float w = tw[j], b = tb[j];
    for (int64_t r = r0 + rg; r < r1; r += 4) {
      float d;
      if (!delta.get(r, d)) continue;
      const float sn = sin_saved ? sin_saved[r * dt_dim + j] : sinf(time_arg(w, d, b));
      const float g = dphi[r * ld + j] * -sn;
      sb += g;
      sw += g * d;
    }
  }
  red_w[rg][threadIdx.x & 63] = sw;
  red_b[rg][threadIdx.x & 63] = sb;
  __syncthreads();
  if (rg == 0 && j < dt_dim) {
    const int c = threadIdx.x;
    part[((int64_t)blockIdx.y * 2 + 0) * dt_dim + j] = ((red_w[0][c] + red_w[1][c]) + red_w[2][c]) + red_w[3][c];
    part[((int64_t)blockIdx.y * 2 + 1) * dt_dim + j] = ((red_b[0][c] + red_b[1][c]) + red_b[2][c]) + red_b[3][c];
  }
}

// One block of 256 threads per column j.  Thread t adds the partials of row chunks t, t + 256, ... in
// that order (loads issued eight at a time, chunks past the count read a valid chunk and add zero);
// chunks beyond the device row count (ceil(rows / chunk_rows)) hold no partial.
__device__ __forceinline__ void timegrad_part(const float* __restrict__ part, int64_t rows,
                                              const int32_t* __restrict__ rows_dev, int chunk_rows, int dt_dim,
                                              float& aw, float& ab) {
  const int j = blockIdx.x, t = threadIdx.x;
  const int64_t nch = cdiv(eff_count(rows, rows_dev), chunk_rows);
  for (int64_t c0 = t; c0 < nch; c0 += 256 * 8) {
    float vw[8], vb[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int64_t c = c0 + 256 * u < nch ? c0 + 256 * u : c0;
      vw[u] = part[(c * 2 + 0) * dt_dim + j];
      vb[u] = part[(c * 2 + 1) * dt_dim + j];
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const bool ok = c0 + 256 * u < nch;
      aw += ok ? vw[u] : 0.f;
      ab += ok ? vb[u] : 0.f;
    }
  }
}

// Block sums of NV values over 256 threads, in a fixed order: a butterfly in each wave (lane 0's
// result), then the four wave sums as (w0 + w1) + (w2 + w3).  s holds 4 NV floats.
template <int NV>
__device__ __forceinline__ void block_sums256(float (&v)[NV], float* s) {
  const int t = threadIdx.x;
#pragma unroll
  for (int i = 0; i < NV; ++i) v[i] = wave_sum(v[i]);
  if ((t & 63) == 0) {
#pragma unroll
    for (int i = 0; i < NV; ++i) s[i * 4 + (t >> 6)] = v[i];
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < NV; ++i) v[i] = (s[i * 4] + s[i * 4 + 1]) + (s[i * 4 + 2] + s[i * 4 + 3]);
}

__global__ __launch_bounds__(256) void k_timegrad_reduce(const float* __restrict__ part, int64_t rows,
                                                         const int32_t* __restrict__ rows_dev, int chunk_rows,
                                                         int dt_dim, float* __restrict__ dw, float* __restrict__ db,
                                                         int accumulate) {
  __shared__ float s[8];
  float v[2] = {0.f, 0.f};
  timegrad_part(part, rows, rows_dev, chunk_rows, dt_dim, v[0], v[1]);
  block_sums256<2>(v, s);
  const int j = blockIdx.x;
  if (threadIdx.x == 0) {
    dw[j] = accumulate ? dw[j] + v[0] : v[0];
    db[j] = accumulate ? db[j] + v[1] : v[1];
  }
}

// The neighbour slots' partial sums plus the queries' share, which is closed-form: a query's time
// input is phi(0) (delta = 0), so its w-gradient is zero and its b-gradient in column j is
// -sin(b_j) sum_i dphi_ij = -sin(b_j) sum_a (sum_i dqv_ia) Wq[a][col0 + j], with sum_i dqv_ia the
// query projection's bias gradient dbq.  The same constant input makes the query weight's time
// columns an outer product, written here too: dWq[a][col0 + j] = dbq[a] phi(0)_j.
__global__ __launch_bounds__(256) void k_timegrad_reduce_q(const float* __restrict__ part, int64_t rows,
                                                           const int32_t* __restrict__ rows_dev, int chunk_rows,
                                                           int dt_dim, const float* __restrict__ dbq,
                                                           const float* __restrict__ Wq, int64_t ldw, int col0, int da,
                                                           const float* __restrict__ tw, const float* __restrict__ tb,
                                                           float* __restrict__ dw, float* __restrict__ db,
                                                           float* __restrict__ dWq) {
  __shared__ float s[12];
  const int j = blockIdx.x, t = threadIdx.x;
  float v[3] = {0.f, 0.f, 0.f};
  const float phi0 = cosf(time_arg(tw[j], 0.f, tb[j]));
  for (int a = t; a < da; a += 256) {
    v[2] += dbq[a] * Wq[(int64_t)a * ldw + col0 + j];
    dWq[(int64_t)a * ldw + col0 + j] = dbq[a] * phi0;
  }
  timegrad_part(part, rows, rows_dev, chunk_rows, dt_dim, v[0], v[1]);
  block_sums256<3>(v, s);
  if (t == 0) {
    dw[j] = v[0];
    db[j] = -sinf(time_arg(tw[j], 0.f, tb[j])) * v[2] + v[1];
  }
}

// Two partial sets in one launch: d = (sum of the first) + (sum of the second), as two reduces
// (the first overwriting, the second accumulating) would give.
__global__ __launch_bounds__(256) void k_timegrad_reduce2(const float* __restrict__ p1, int64_t rows1,
                                                          const int32_t* __restrict__ rows_dev1,
                                                          const float* __restrict__ p2, int64_t rows2,
                                                          const int32_t* __restrict__ rows_dev2, int chunk_rows,
                                                          int dt_dim, float* __restrict__ dw, float* __restrict__ db) {
  __shared__ float s[16];
  float v[4] = {0.f, 0.f, 0.f, 0.f};
  timegrad_part(p1, rows1, rows_dev1, chunk_rows, dt_dim, v[0], v[1]);
  timegrad_part(p2, rows2, rows_dev2, chunk_rows, dt_dim, v[2], v[3]);
  block_sums256<4>(v, s);
  const int j = blockIdx.x;
  if (threadIdx.x == 0) {
    dw[j] = v[0] + v[2];
    db[j] = v[1] + v[3];
  }
}

}  // namespace

// ---------------------------------------------------------------- shared time-grad launcher

size_t timegrad_ws_bytes(int64_t rows, int dt_dim) {
  return a256(sizeof(float) * 2 * (size_t)cdiv(rows < 1 ? 1 : rows, TG_ROWS) * dt_dim);
}

template <typename D>
mtgnn_status timegrad_launch(const float* dphi, int64_t ld, int64_t rows, const int32_t* rows_dev, D delta,
                             const float* tw, const float* tb, const float* sin_saved, int dt_dim, float* dw, float* db,
                             bool accumulate, void* ws, size_t ws_bytes, hipStream_t s) {
  if (dt_dim <= 0) return MTGNN_OK;
  if (rows <= 0) rows = 1;   // still writes (zero) sums when overwriting
  if (ws_bytes < timegrad_ws_bytes(rows, dt_dim)) return MTGNN_EWORKSPACE;
  const int nch = (int)cdiv(rows, TG_ROWS);
  dim3 g((unsigned)cdiv(dt_dim, 64), (unsigned)nch);
  k_timegrad_partial<D><<<g, 256, 0, s>>>(dphi, ld, rows, rows_dev, delta, tw, tb, sin_saved, dt_dim, (float*)ws);
  MTGNN_CHECK_LAUNCH("timegrad_partial");
k_timegrad_reduce<<<(unsigned)dt_dim, 256, 0, s>>>((const float*)ws, rows, rows_dev, TG_ROWS, dt_dim, dw, db,
                                                     accumulate ? 1 : 0);
  MTGNN_CHECK_LAUNCH("timegrad_reduce");
  return MTGNN_OK;
}

mtgnn_status timegrad_reduce_blocks(const float* part, int64_t rows, const int32_t* rows_dev, int chunk_rows,
                                    int dt_dim, float* dw, float* db, bool accumulate, hipStream_t s) {
  if (dt_dim <= 0) return MTGNN_OK;
  k_timegrad_reduce<<<(unsigned)dt_dim, 256, 0, s>>>(part, rows, rows_dev, chunk_rows, dt_dim, dw, db,
                                                      accumulate ? 1 : 0);
  MTGNN_CHECK_LAUNCH("timegrad_reduce");
  return MTGNN_OK;
}

mtgnn_status timegrad_reduce_slots_q(const float* part, int64_t rows, const int32_t* rows_dev, int chunk_rows,
                                     int dt_dim, const float* dbq, const float* Wq, int64_t ldw, int col0, int da,
                                     const float* tw, const float* tb, float* dw, float* db, float* dWq,
                                     hipStream_t s) {
  if (dt_dim <= 0) return MTGNN_OK;
  k_timegrad_reduce_q<<<(unsigned)dt_dim, 256, 0, s>>>(part, rows, rows_dev, chunk_rows, dt_dim, dbq, Wq, ldw, col0,
                                                        da, tw, tb, dw, db, dWq);
  MTGNN_CHECK_LAUNCH("timegrad_reduce_q");
  return MTGNN_OK;
}

mtgnn_status timegrad_reduce_blocks2(const float* p1, int64_t rows1, const int32_t* rows_dev1, const float* p2,
                                     int64_t rows2, const int32_t* rows_dev2, int chunk_rows, int dt_dim, float* dw,
                                     float* db, hipStream_t s) {
  if (dt_dim <= 0) return MTGNN_OK;
  k_timegrad_reduce2<<<(unsigned)dt_dim, 256, 0, s>>>(p1, rows1, rows_dev1, p2, rows2, rows_dev2, chunk_rows, dt_dim,
                                                       dw, db);
  MTGNN_CHECK_LAUNCH("timegrad_reduce2");
  return MTGNN_OK;
}

mtgnn_status timegrad_rows(const float* dphi, int64_t ld, int64_t rows, const int32_t* rows_dev, const float* delta,
                           const float* sin_saved, const float* tw, const float* tb, int dt_dim, float* dw, float* db,
                           bool accumulate, void* ws, size_t ws_bytes, hipStream_t s) {
  return timegrad_launch(dphi, ld, rows, rows_dev, RowDelta{delta}, tw, tb, sin_saved, dt_dim, dw, db, accumulate, ws,
                         ws_bytes, s);
}

// ---------------------------------------------------------------- entry-point bodies

size_t build_queries_ws(int64_t n) { return 2 * a256(sizeof(int32_t) * n) + a256(sizeof(int32_t)) + scan_ws_bytes(n); }

mtgnn_status build_queries_impl(const mtgnn_batch* b, const int32_t* neg, int32_t* q_node, float* q_t, int32_t* n_q,
                                void* ws, size_t ws_bytes, hipStream_t s) {
  const int64_t n = b->n;
  if (b->flags == nullptr || n == 0) {
    k_queries_all<<<(unsigned)cdiv(n < 1 ? 1 : n, 256), 256, 0, s>>>(b->src, b->dst, neg, b->t, n, q_node, q_t, n_q);
    MTGNN_CHECK_LAUNCH("queries_all");
    return MTGNN_OK;
  }
  if (ws_bytes < build_queries_ws(n)) return MTGNN_EWORKSPACE;
  char* w = (char*)ws;
  int32_t* tgt = (int32_t*)w;
  w += a256(sizeof(int32_t) * n);
  int32_t* pos = (int32_t*)w;
  w += a256(sizeof(int32_t) * n);
  int32_t* ntar = (int32_t*)w;
  w += a256(sizeof(int32_t));
  const unsigned grid = (unsigned)cdiv(n, 256);
  k_target_flags<<<grid, 256, 0, s>>>(b->flags, n, tgt);
  MTGNN_CHECK_LAUNCH("target_flags");
  MTGNN_TRY(scan_exclusive(tgt, pos, n, ntar, w, ws_bytes - (size_t)(w - (char*)ws), s));
  k_queries_masked<<<grid, 256, 0, s>>>(b->src, b->dst, neg, b->t, b->flags, n, pos, ntar, q_node, q_t, n_q);
  MTGNN_CHECK_LAUNCH("queries_masked");
  return MTGNN_OK;
}

size_t aggregate_last_ws(int64_t n, int64_t n_nodes) {
  const int64_t nm = 2 * n;
  size_t b = a256(sizeof(int32_t) * (n_nodes > 0 ? n_nodes : 1));
  if (nm > AGG_BLOCK_MAX) b += 2 * a256(sizeof(int32_t) * nm) + scan_ws_bytes(nm);
  return b;
}

mtgnn_status aggregate_last_impl(const mtgnn_batch* b, int64_t n_nodes, int32_t* uniq, int32_t* winner,
                                 int32_t* n_uniq, void* ws, size_t ws_bytes, hipStream_t s) {
  const int64_t n = b->n, nm = 2 * n;
  if (n == 0) {
    k_set_int<<<1, 1, 0, s>>>(n_uniq, 0);
    MTGNN_CHECK_LAUNCH("set_int");
    return MTGNN_OK;
  }
  if (ws_bytes < aggregate_last_ws(n, n_nodes)) return MTGNN_EWORKSPACE;
  char* w = (char*)ws;
  int32_t* T = (int32_t*)w;
  w += a256(sizeof(int32_t) * n_nodes);
  const unsigned grid = (unsigned)cdiv(nm, 256);
  k_agg_reset<<<grid, 256, 0, s>>>(b->src, b->dst, b->flags, nm, T);
  MTGNN_CHECK_LAUNCH("agg_reset");
  k_agg_max<<<grid, 256, 0, s>>>(b->src, b->dst, b->flags, nm, T);
  MTGNN_CHECK_LAUNCH("agg_max");
  if (nm <= AGG_BLOCK_MAX) {
    k_agg_compact_block<<<1, AGG_BLOCK_THREADS, 0, s>>>(b->src, b->dst, b->flags, nm, T, uniq, winner, n_uniq);
    MTGNN_CHECK_LAUNCH("agg_compact_block");
    return MTGNN_OK;
  }
  int32_t* win = (int32_t*)w;
  w += a256(sizeof(int32_t) * nm);
  int32_t* pos = (int32_t*)w;
  w += a256(sizeof(int32_t) * nm);
  const size_t rest = ws_bytes - (size_t)(w - (char*)ws);
  k_agg_flags<<<grid, 256, 0, s>>>(b->src, b->dst, b->flags, nm, T, win);
  MTGNN_CHECK_LAUNCH("agg_flags");
  MTGNN_TRY(scan_exclusive(win, pos, nm, n_uniq, w, rest, s));
  k_agg_write<<<grid, 256, 0, s>>>(b->src, b->dst, b->flags, nm, win, pos, uniq, winner);
  MTGNN_CHECK_LAUNCH("agg_write");
  return MTGNN_OK;
}

mtgnn_status build_messages_impl(const mtgnn_batch* b, const int32_t* uniq, const int32_t* winner,
                                 const int32_t* n_rows, int64_t max_rows, const void* memory, const float* lu,
                                 const float* edge_feat, const float* tw, const float* tb, const mtgnn_dims* d,
                                 void* msg, float* dt, hipStream_t s) {
  const unsigned grid = (unsigned)cdiv(max_rows, 4);
  if (d->dtype == MTGNN_F32)
    k_build_messages<float><<<grid, 256, 0, s>>>(b->src, b->dst, b->eid, b->t, uniq, winner, n_rows, max_rows,
                                                  (const float*)memory, lu, edge_feat, tw, tb, d->d_mem, d->d_time,
                                                  d->d_edge, (float*)msg, dt);
  else
    k_build_messages<uint16_t><<<grid, 256, 0, s>>>(b->src, b->dst, b->eid, b->t, uniq, winner, n_rows, max_rows,
                                                     (const uint16_t*)memory, lu, edge_feat, tw, tb, d->d_mem,
                                                     d->d_time, d->d_edge, (uint16_t*)msg, dt);
  MTGNN_CHECK_LAUNCH("build_messages");
  return MTGNN_OK;
}

// GRU save layout: h_old, r, z, n, ghn, each [max_rows, d_mem] float32, then (float32) the padded
// W_ih[:, 2 dm : 2 dm + dt]^T of the backward's fused time-feature gradient.  In float32 the h_old plane
// stays unused: the message rows start with M[uniq[r]] (the same values), so both passes read h
// from msg with its row stride instead of gathering it.
size_t gru_save_bytes(const mtgnn_dims* d, int64_t max_rows) {
  const size_t wt = gru_dx_fused_ok(d->dtype, d->d_mem, d->d_time) ? gru_dx_weight_floats(d->d_mem, d->d_time) : 1;
  return 5 * a256(sizeof(float) * max_rows * d->d_mem) + a256(sizeof(float) * wt);
}

size_t gru_update_ws(const mtgnn_dims* d, int64_t max_rows) {
  const int dmsg = 2 * d->d_mem + d->d_time + d->d_edge;
  return a256(sizeof(float) * max_rows * 6 * d->d_mem) + a256(sizeof(float) * max_rows * d->d_mem) +
         a256(sizeof(float) * gru_fused_weight_floats(d->d_mem, dmsg));
}

mtgnn_status gru_update_impl(const mtgnn_batch* b, const int32_t* uniq, const int32_t* winner, const int32_t* n_rows,
                             int64_t max_rows, const void* msg, const void* W_ih, const void* W_hh, const float* b_ih,
                             const float* b_hh, const mtgnn_dims* d, void* memory, float* lu, void* save, void* ws,
                             size_t ws_bytes, hipStream_t s) {
  if (ws_bytes < gru_update_ws(d, max_rows)) return MTGNN_EWORKSPACE;
  const int dm = d->d_mem, dmsg = 2 * d->d_mem + d->d_time + d->d_edge;
  const size_t plane = a256(sizeof(float) * max_rows * dm);
  float* G = (float*)ws;
  float* h_old = save ? (float*)save : (float*)((char*)ws + a256(sizeof(float) * max_rows * 6 * dm));
  float *sr = nullptr, *sz = nullptr, *sn = nullptr, *sghn = nullptr;
  if (save) {
    sr = (float*)((char*)save + plane);
    sz = (float*)((char*)save + 2 * plane);
    sn = (float*)((char*)save + 3 * plane);
    sghn = (float*)((char*)save + 4 * plane);
  }
  const unsigned gel = (unsigned)cdiv(max_rows * dm, 256);
  int64_t ldh = dm;
  if (gru_fused_ok(d->dtype, dm, dmsg)) {   // both products and the gates in one kernel
    GruWTArgs wa{};
    if (save && gru_dx_fused_ok(d->dtype, dm, d->d_time)) {
      const int kc = (int)cdiv(3 * dm, 16);
      wa = GruWTArgs{(float*)((char*)save + 5 * plane), (int)(gru_dx_weight_floats(dm, d->d_time) / (16 * kc)),
                     16 * kc, d->d_time, 3 * dm, dmsg, 2 * dm};
    }
    float* Wp = (float*)((char*)ws + a256(sizeof(float) * max_rows * 6 * dm) + a256(sizeof(float) * max_rows * dm));
    return gru_fused((const float*)msg, (const float*)W_ih, (const float*)W_hh, b_ih, b_hh, uniq, winner, b->t,
                     n_rows, max_rows, dm, dmsg, Wp, (float*)memory, lu, sr, sz, sn, sghn, wa, s);
  }
  if (d->dtype == MTGNN_F32) {   // h = msg[:, :dm]; both products in one launch (their inputs share a type)
    h_old = (float*)msg;
    ldh = dmsg;
    const FwdProblem ps[2] = {{msg, dmsg, W_ih, dmsg, b_ih, G, 6 * dm, 3 * dm, dmsg},
                              {msg, dmsg, W_hh, dm, b_hh, G + 3 * dm, 6 * dm, 3 * dm, dm}};
    MTGNN_TRY(linear_fwd_batch(ps, 2, max_rows, n_rows, MTGNN_F32, MTGNN_F32, s));
  } else {
    k_gather_rows<uint16_t><<<gel, 256, 0, s>>>((const uint16_t*)memory, uniq, n_rows, max_rows, dm, h_old);
    MTGNN_CHECK_LAUNCH("gather_rows");
    MTGNN_TRY(linear_fwd(msg, d->dtype, dmsg, W_ih, d->dtype, dmsg, b_ih, G, 6 * dm, max_rows, n_rows, 3 * dm, dmsg,
                         false, s));
    MTGNN_TRY(linear_fwd(h_old, MTGNN_F32, dm, W_hh, d->dtype, dm, b_hh, G + 3 * dm, 6 * dm, max_rows, n_rows, 3 * dm,
                         dm, false, s));
  }
  GruWT wt{};
  if (save && gru_dx_fused_ok(d->dtype, dm, d->d_time)) {
    const int kc = (int)cdiv(3 * dm, 16);
    wt = GruWT{(const float*)W_ih, (float*)((char*)save + 5 * plane),
               (int)(gru_dx_weight_floats(dm, d->d_time) / (16 * kc)), 16 * kc, d->d_time, 3 * dm, dmsg, 2 * dm};
  }
  if (d->dtype == MTGNN_F32)
    k_gru_gates<float><<<gel, 256, 0, s>>>(G, h_old, ldh, uniq, winner, b->t, n_rows, max_rows, dm, (float*)memory,
                                           lu, sr, sz, sn, sghn, wt);
  else
    k_gru_gates<uint16_t><<<gel, 256, 0, s>>>(G, h_old, ldh, uniq, winner, b->t, n_rows, max_rows, dm,
                                              (uint16_t*)memory, lu, sr, sz, sn, sghn, wt);
  MTGNN_CHECK_LAUNCH("gru_gates");
  return MTGNN_OK;
}

// The float32 GRU weight gradients as output tiles (dw_tiles).  The reset and update gates' hidden
// products equal their input products over the message's first d_mem columns (h is that slice and both
// products see the same pre-activation gradient), so dW_hh's r, z rows and db_hh's r, z entries are
// copies of dW_ih's and db_ih's: only the candidate's hidden product is computed apart.
//   dW_ih = dgi^T [msg | 1]: column tiles of the 3 d_mem gradient columns (<= 112 wide) times column tiles
//   of the message ([0, d_mem), then <= 108 wide); dW_hh,n = dgh_n^T [h | 1].
// Returns the tile count, 0 if the shape does not fit.
static int gru_dw_tiles(const float* dgi, const float* dgh, const float* msg, int dm, int dmsg, float* dW_ih,
                        float* dW_hh, float* db_ih, float* db_hh, DwTile* t) {
  if (dm % 4 || dmsg % 4 || dm > 108 || dmsg <= dm) return 0;
  const int nxt = (int)cdiv(3 * dm, 112), wx = (int)cdiv(cdiv(3 * dm, nxt), 4) * 4;
  const int nyt = (int)cdiv(dmsg - dm, 108), wy = (int)cdiv(cdiv(dmsg - dm, nyt), 4) * 4;
  if (nxt * (nyt + 1) + 1 > DW_OS_MAXP) return 0;
  int n = 0;
  for (int x0 = 0; x0 < 3 * dm; x0 += wx) {
    const int nx = std::min(wx, 3 * dm - x0);
    const int shared = std::max(0, std::min(nx, 2 * dm - x0));   // reset and update rows of this tile
    for (int y0 = 0; y0 < dmsg; y0 = y0 == 0 ? dm : y0 + wy) {
      const int ny = y0 == 0 ? dm : std::min(wy, dmsg - y0);
      const bool last = y0 + ny == dmsg;
      DwTile q{};
      q.X = dgi + x0;
      q.ldx = 3 * dm;
      q.Y = msg + y0;
      q.ldy = dmsg;
      q.nx = nx;
      q.ny = ny;
      q.dW = dW_ih + (int64_t)x0 * dmsg + y0;
      q.lddw = dmsg;
      q.db = last ? db_ih + x0 : nullptr;
      if (shared > 0 && (y0 == 0 || last)) {
        q.dup = y0 == 0 ? dW_hh + (int64_t)x0 * dm : nullptr;
        q.lddup = dm;
        q.dup_rows = shared;
        q.dup_db = last ? db_hh + x0 : nullptr;
      }
      t[n++] = q;
    }
  }
  DwTile q{};
  q.X = dgh + 2 * dm;
  q.ldx = 3 * dm;
  q.Y = msg;
  q.ldy = dmsg;
  q.nx = q.ny = dm;
  q.dW = dW_hh + (int64_t)2 * dm * dm;
  q.lddw = dm;
  q.db = db_hh + 2 * dm;
  t[n++] = q;
  return n;
}

size_t gru_update_bwd_ws(const mtgnn_dims* d, int64_t max_rows) {
  const int dm = d->d_mem, dmsg = 2 * d->d_mem + d->d_time + d->d_edge;
  size_t dw = linear_dw_ws_bytes(max_rows, 3 * dm, dmsg);
  size_t dw2 = linear_dw_ws_bytes(max_rows, 3 * dm, dm);
  const int64_t Ns[2] = {3 * dm, 3 * dm}, Ks[2] = {dmsg, dm};
  size_t dwb = linear_dw_batch_ws_bytes(max_rows, Ns, Ks, 2);
  size_t m = dw > dw2 ? dw : dw2;
  m = m > dwb ? m : dwb;
  DwTile t[DW_OS_MAXP];
  const float* base = nullptr;   // tile offsets only: the sizes do not depend on the buffers
  const int nt = d->dtype == MTGNN_F32 ? gru_dw_tiles(base, base, base, dm, dmsg, nullptr, nullptr, nullptr,
                                                      nullptr, t) : 0;
  if (nt) m = std::max(m, dw_tiles_ws_bytes(t, nt));
  return 2 * a256(sizeof(float) * max_rows * 3 * dm) + a256(m);
}

mtgnn_status gru_update_bwd_impl(const float* d_mem, const void* save, const void* msg, const int32_t* n_rows,
                                 int64_t max_rows, const void* W_ih, const void* W_hh, const mtgnn_dims* d, float* dW_ih,
                                 float* dW_hh, float* db_ih, float* db_hh, float* dmsg_time, void* ws, size_t ws_bytes,
                                 hipStream_t s) {
  if (ws_bytes < gru_update_bwd_ws(d, max_rows)) return MTGNN_EWORKSPACE;
  const int dm = d->d_mem, dmsg = 2 * d->d_mem + d->d_time + d->d_edge;
  const size_t plane = a256(sizeof(float) * max_rows * dm);
  const bool f32 = d->dtype == MTGNN_F32;
  const float* h_old = f32 ? (const float*)msg : (const float*)save;   // float32: h = msg[:, :dm]
  const int64_t ldh = f32 ? dmsg : dm;
  const float* sr = (const float*)((const char*)save + plane);
  const float* sz = (const float*)((const char*)save + 2 * plane);
  const float* sn = (const float*)((const char*)save + 3 * plane);
  const float* sghn = (const float*)((const char*)save + 4 * plane);
  char* w = (char*)ws;
  float* dgi = (float*)w;
  w += a256(sizeof(float) * max_rows * 3 * dm);
  float* dgh = (float*)w;
  w += a256(sizeof(float) * max_rows * 3 * dm);
  const size_t rest = ws_bytes - (size_t)(w - (char*)ws);
  k_gru_bwd_gates<<<(unsigned)cdiv(max_rows * dm, 256), 256, 0, s>>>(d_mem, h_old, ldh, sr, sz, sn, sghn, n_rows,
                                                                        max_rows, dm, dgi, dgh);
  MTGNN_CHECK_LAUNCH("gru_bwd_gates");
  DwTile tiles[DW_OS_MAXP];
  const int nt = d->dtype == MTGNN_F32 ? gru_dw_tiles(dgi, dgh, (const float*)msg, dm, dmsg, dW_ih, dW_hh, db_ih,
                                                      db_hh, tiles) : 0;
  mtgnn_status st = MTGNN_EUNSUPPORTED;
  if (nt) {   // one output-stationary launch and one reduce (unsupported: misaligned operands)
    TimedScope ts(site::GruDw::name, s);
    st = dw_tiles<site::GruDw>(tiles, nt, max_rows, n_rows, w, rest, s);
    if (st != MTGNN_OK && st != MTGNN_EUNSUPPORTED) return st;
  }
  if (st != MTGNN_OK && d->dtype == MTGNN_F32) {   // both weight gradients in one launch
    const DwProblem ps[2] = {{dgi, 3 * dm, msg, dmsg, dW_ih, dmsg, 3 * dm, dmsg, db_ih},
                             {dgh, 3 * dm, h_old, ldh, dW_hh, dm, 3 * dm, dm, db_hh}};
    MTGNN_TRY(linear_dw_batch<site::GruDw>(ps, 2, max_rows, n_rows, MTGNN_F32, w, rest, s));
  } else if (st != MTGNN_OK) {
    MTGNN_TRY(linear_dw(dgi, 3 * dm, msg, d->dtype, dmsg, dW_ih, dmsg, max_rows, n_rows, 3 * dm, dmsg, w, rest, s,
                        db_ih));
    MTGNN_TRY(linear_dw(dgh, 3 * dm, h_old, MTGNN_F32, dm, dW_hh, dm, max_rows, n_rows, 3 * dm, dm, w, rest, s,
                        db_hh));
  }
  if (dmsg_time && d->d_time > 0 && gru_dx_fused_ok(d->dtype, dm, d->d_time))
    return gru_dx_fused(dgi, (const float*)((const char*)save + 5 * plane), dmsg_time, n_rows, max_rows, dm,
                        d->d_time, s);
  if (dmsg_time && d->d_time > 0) {
    const size_t esz = d->dtype == MTGNN_F32 ? 4 : 2;
    const void* Wt = (const char*)W_ih + esz * (size_t)(2 * dm);   // columns [2 dm, 2 dm + d_time)
    MTGNN_TRY(linear_dx(dgi, 3 * dm, Wt, d->dtype, dmsg, dmsg_time, d->d_time, max_rows, n_rows, 3 * dm, d->d_time,
                        false, s));
  }
  return MTGNN_OK;
}

size_t build_messages_bwd_ws(const mtgnn_dims* d, int64_t max_rows) { return timegrad_ws_bytes(max_rows, d->d_time); }

mtgnn_status build_messages_bwd_impl(const float* dmsg_time, const float* dt, const int32_t* n_rows, int64_t max_rows,
                                     const float* tw, const float* tb, const mtgnn_dims* d, float* dw, float* db,
                                     void* ws, size_t ws_bytes, hipStream_t s) {
  return timegrad_rows(dmsg_time, d->d_time, max_rows, n_rows, dt, nullptr, tw, tb, d->d_time, dw, db, true, ws,
                       ws_bytes, s);
}

}  // namespace mtgnn

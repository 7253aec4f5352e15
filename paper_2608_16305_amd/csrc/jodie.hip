// The JODIE variant of the batch step (Section VII-A): a recurrent memory update and a time-projection
// embedding, on the same aggregation, messages and masked link loss as TGN.
//   update:      h' = tanh(W_ih x + b_ih + W_hh h + b_hh), x = the winning message, h = M[node]
//                (the first d_mem columns of the message, so the hidden product reads the message rows);
//   embedding:   z = M[n] (1 + W_p Delta + b_p), Delta = (tau - last_update[n]) s;
//   backward:    dW_p, db_p as fixed-order column sums; d M' for the updated rows as fixed-order sums over
//                each row's query occurrences (stable sort of the occurrences by updated row); the
//                update's gradients through dpre = d M' (1 - h'^2).
#include "gemm.h"
#include "ops.h"

namespace mtgnn {

namespace {

size_t a256j(size_t x) { return (x + 255) & ~size_t(255); }

// G [max_rows, 2 dm]: the input and hidden products (with their biases); wave per row.
template <typename T>
__global__ __launch_bounds__(256) void k_rnn_act(const float* __restrict__ G, const int32_t* __restrict__ uniq,
                                                 const int32_t* __restrict__ winner, const float* __restrict__ t,
                                                 const int32_t* __restrict__ n_rows, int64_t max_rows, int dm,
                                                 T* __restrict__ mem, float* __restrict__ lu,
                                                 float* __restrict__ save_h) {
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= eff_count(max_rows, n_rows)) return;
  const int64_t node = uniq[r];
  for (int j = lane; j < dm; j += 64) {
    const float h = tanhf(G[r * 2 * dm + j] + G[r * 2 * dm + dm + j]);
    Elem<T>::store(mem, node * dm + j, h);
    if (save_h) save_h[r * dm + j] = h;
  }
  if (lane == 0) lu[node] = t[winner[r] >> 1];
}

__global__ void k_rnn_dpre(const float* __restrict__ d_mem, const float* __restrict__ h,
                           const int32_t* __restrict__ n_rows, int64_t max_rows, int dm, float* __restrict__ dp) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t R = eff_count(max_rows, n_rows);
  if (i >= R * dm) return;
  const float v = h[i];
  dp[i] = d_mem[i] * (1.0f - v * v);
}

template <typename T>
__device__ __forceinline__ float proj_delta(const float* q_t, const float* lu, int64_t q, int64_t n, float s) {
  const float d = q_t[q] - lu[n];
  return d * s;
}

// z = M[n] (1 + W_p Delta + b_p); wave per query.
template <typename T>
__global__ __launch_bounds__(256) void k_time_proj(const int32_t* __restrict__ q_node, const float* __restrict__ q_t,
                                                   const int32_t* __restrict__ n_q, int64_t max_q,
                                                   const T* __restrict__ mem, const float* __restrict__ lu,
                                                   const float* __restrict__ Wp, const float* __restrict__ bp,
                                                   float s, int dm, float* __restrict__ z) {
  const int64_t q = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (q >= eff_count(max_q, n_q)) return;
  const int64_t n = q_node[q];
  const float dl = proj_delta<T>(q_t, lu, q, n, s);
  for (int j = lane; j < dm; j += 64) z[q * dm + j] = Elem<T>::load(mem, n * dm + j) * (1.0f + dl * Wp[j] + bp[j]);
}

// Per query: G[q] = [dz M Delta | dz M] (for the column sums of dW_p, db_p), and the occurrence key of its
// node (its updated row, or the sentinel max_rows).
template <typename T>
__global__ __launch_bounds__(256) void k_time_proj_bwd_rows(
    const int32_t* __restrict__ q_node, const float* __restrict__ q_t, const int32_t* __restrict__ n_q, int64_t max_q,
    const T* __restrict__ mem, const float* __restrict__ lu, float s, int dm, const float* __restrict__ dz,
    const int32_t* __restrict__ uniq, const int32_t* __restrict__ n_rows, const int32_t* __restrict__ row_of,
    int64_t max_rows, const float* __restrict__ Wp, const float* __restrict__ bp, float* __restrict__ G,
    float* __restrict__ Cq, uint32_t* __restrict__ keys, uint32_t* __restrict__ vals) {
  const int64_t q = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (q >= max_q) return;
  const bool live = q < eff_count(max_q, n_q);
  if (lane == 0) {
    uint32_t key = (uint32_t)max_rows;
    if (live) {
      const int32_t n = q_node[q];
      const int32_t r = row_of[n];
      if (r >= 0 && r < eff_count(max_rows, n_rows) && uniq[r] == n) key = (uint32_t)r;
    }
    keys[q] = key;
    vals[q] = (uint32_t)q;
  }
  if (!live) {
    for (int j = lane; j < 2 * dm; j += 64) G[q * 2 * dm + j] = 0.f;
    return;
  }
  const int64_t n = q_node[q];
  const float dl = proj_delta<T>(q_t, lu, q, n, s);
  for (int j = lane; j < dm; j += 64) {
    const float g = dz[q * dm + j] * Elem<T>::load(mem, n * dm + j);
    G[q * 2 * dm + j] = g * dl;
    G[q * 2 * dm + dm + j] = g;
    Cq[q * dm + j] = dz[q * dm + j] * (1.0f + dl * Wp[j] + bp[j]);
  }
}

// row_of[uniq[r]] = r for the updated rows (entries of other nodes are stale and are rejected on use).
__global__ void k_jodie_row_map(const int32_t* __restrict__ uniq, const int32_t* __restrict__ n_rows, int64_t max_rows,
                                int32_t* __restrict__ row_of) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r < eff_count(max_rows, n_rows)) row_of[uniq[r]] = (int32_t)r;
}

__device__ __forceinline__ int64_t lower_bound_u32(const uint32_t* k, int64_t n, uint32_t v) {
  int64_t lo = 0, hi = n;
  while (lo < hi) {
    const int64_t mid = (lo + hi) >> 1;
    if (k[mid] < v) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

// d M'[r] = sum over row r's query occurrences (stable order) of dz[q] (1 + W_p Delta_q + b_p); wave per row.
template <typename T>
__global__ __launch_bounds__(256) void k_jodie_dmem(const uint32_t* __restrict__ skeys, const uint32_t* __restrict__ svals,
                                                    int64_t n_occ, const int32_t* __restrict__ q_node,
                                                    const float* __restrict__ q_t, const float* __restrict__ lu,
                                                    const float* __restrict__ Wp, const float* __restrict__ bp, float s,
                                                    const float* __restrict__ dz, const int32_t* __restrict__ n_rows,
                                                    int64_t max_rows, int dm, float* __restrict__ d_mem) {
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= eff_count(max_rows, n_rows)) return;
  const int64_t lo = lower_bound_u32(skeys, n_occ, (uint32_t)r);
  const int64_t hi = lower_bound_u32(skeys, n_occ, (uint32_t)r + 1);
  constexpr int NC = 4;   // columns per lane: d_mem <= 256
  float acc[NC] = {0.f, 0.f, 0.f, 0.f};
  for (int64_t i = lo; i < hi; ++i) {
    const int64_t q = svals[i];
    const float dl = proj_delta<T>(q_t, lu, q, q_node[q], s);
#pragma unroll
    for (int u = 0; u < NC; ++u) {
      const int j = lane + 64 * u;
      if (j < dm) acc[u] += dz[q * dm + j] * (1.0f + dl * Wp[j] + bp[j]);
    }
  }
#pragma unroll
  for (int u = 0; u < NC; ++u) {
    const int j = lane + 64 * u;
    if (j < dm) d_mem[r * dm + j] = acc[u];
  }
}

// The same sums with the occurrences spread over the lanes: lane l adds occurrences l, l + 64, ... of the
// row's segment (all d_mem columns, 4 per register group), then the 64 lane sums are added by a fixed
// butterfly per column.  A hub row's thousands of occurrences then take tens of rounds, not thousands.
template <int NQ>
__global__ __launch_bounds__(256) void k_jodie_dmem_lanes(const uint32_t* __restrict__ skeys,
                                                          const uint32_t* __restrict__ svals, int64_t n_occ,
                                                          const float* __restrict__ Cq,
                                                          const int32_t* __restrict__ n_rows, int64_t max_rows, int dm,
                                                          float* __restrict__ d_mem) {
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= eff_count(max_rows, n_rows)) return;
  const int64_t lo = lower_bound_u32(skeys, n_occ, (uint32_t)r);
  const int64_t hi = lower_bound_u32(skeys, n_occ, (uint32_t)r + 1);
  float4 acc[NQ];
#pragma unroll
  for (int u = 0; u < NQ; ++u) acc[u] = float4{0.f, 0.f, 0.f, 0.f};
  const int nq = dm / 4;
  for (int64_t i = lo + lane; i < hi; i += 64) {
    const float4* row = reinterpret_cast<const float4*>(Cq + (int64_t)svals[i] * dm);
#pragma unroll
    for (int u = 0; u < NQ; ++u) {
      if (u < nq) {
        const float4 c = row[u];
        acc[u].x += c.x;
        acc[u].y += c.y;
        acc[u].z += c.z;
        acc[u].w += c.w;
      }
    }
  }
#pragma unroll
  for (int u = 0; u < NQ; ++u) {
    if (u < nq) {
      const float x = wave_sum(acc[u].x), y = wave_sum(acc[u].y), z = wave_sum(acc[u].z), w = wave_sum(acc[u].w);
      if (lane == 0) reinterpret_cast<float4*>(d_mem + r * dm)[u] = float4{x, y, z, w};
    }
  }
}

__global__ void k_split_sums(const float* __restrict__ sums, int dm, float* __restrict__ dWp, float* __restrict__ dbp) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j < dm) {
    dWp[j] = sums[j];
    dbp[j] = sums[dm + j];
  }
}

}  // namespace

// ---------------------------------------------------------------- recurrent update

size_t rnn_save_bytes(const mtgnn_dims* d, int64_t max_rows) { return a256j(sizeof(float) * (size_t)max_rows * d->d_mem); }
size_t rnn_update_ws(const mtgnn_dims* d, int64_t max_rows) {
  return a256j(sizeof(float) * (size_t)(max_rows < 1 ? 1 : max_rows) * 2 * d->d_mem);
}

mtgnn_status rnn_update_impl(const mtgnn_batch* b, const int32_t* uniq, const int32_t* winner, const int32_t* n_rows,
                             int64_t max_rows, const void* msg, const void* W_ih, const void* W_hh, const float* b_ih,
                             const float* b_hh, const mtgnn_dims* d, void* memory, float* lu, void* save, void* ws,
                             size_t ws_bytes, hipStream_t s) {
  if (max_rows <= 0) return MTGNN_OK;
  if (ws_bytes < rnn_update_ws(d, max_rows)) return MTGNN_EWORKSPACE;
  const int dm = d->d_mem, dmsg = 2 * d->d_mem + d->d_time + d->d_edge;
  float* G = (float*)ws;
  const FwdProblem ps[2] = {{msg, dmsg, W_ih, dmsg, b_ih, G, 2 * dm, dm, dmsg},
                            {msg, dmsg, W_hh, dm, b_hh, G + dm, 2 * dm, dm, dm}};
  MTGNN_TRY(linear_fwd_batch(ps, 2, max_rows, n_rows, d->dtype, d->dtype, s));
  const unsigned g = (unsigned)cdiv(max_rows, 4);
  if (d->dtype == MTGNN_BF16)
    k_rnn_act<uint16_t><<<g, 256, 0, s>>>(G, uniq, winner, b->t, n_rows, max_rows, dm, (uint16_t*)memory, lu,
                                          (float*)save);
  else
    k_rnn_act<float><<<g, 256, 0, s>>>(G, uniq, winner, b->t, n_rows, max_rows, dm, (float*)memory, lu,
                                       (float*)save);
  MTGNN_CHECK_LAUNCH("rnn_act");
  return MTGNN_OK;
}

size_t rnn_update_bwd_ws(const mtgnn_dims* d, int64_t max_rows) {
  const int64_t dm = d->d_mem, dmsg = 2 * d->d_mem + d->d_time + d->d_edge;
  const int64_t N[2] = {dm, dm}, K[2] = {dmsg, dm};
  return a256j(sizeof(float) * (size_t)(max_rows < 1 ? 1 : max_rows) * dm) +
         linear_dw_batch_ws_bytes(max_rows, N, K, 2);
}

mtgnn_status rnn_update_bwd_impl(const float* d_mem, const void* save, const void* msg, const int32_t* n_rows,
                                 int64_t max_rows, const void* W_ih, const void* W_hh, const mtgnn_dims* d,
                                 float* dW_ih, float* dW_hh, float* db_ih, float* db_hh, float* dmsg_time, void* ws,
                                 size_t ws_bytes, hipStream_t s) {
  if (ws_bytes < rnn_update_bwd_ws(d, max_rows)) return MTGNN_EWORKSPACE;
  const int dm = d->d_mem, dmsg = 2 * d->d_mem + d->d_time + d->d_edge;
  float* DP = (float*)ws;
  char* rest = (char*)ws + a256j(sizeof(float) * (size_t)(max_rows < 1 ? 1 : max_rows) * dm);
  k_rnn_dpre<<<(unsigned)cdiv(max_rows * dm, 256), 256, 0, s>>>(d_mem, (const float*)save, n_rows, max_rows, dm, DP);
  MTGNN_CHECK_LAUNCH("rnn_dpre");
  const DwProblem ps[2] = {{DP, dm, msg, dmsg, dW_ih, dmsg, dm, dmsg, db_ih},
                           {DP, dm, msg, dmsg, dW_hh, dm, dm, dm, db_hh}};
  MTGNN_TRY(linear_dw_batch(ps, 2, max_rows, n_rows, d->dtype, rest, ws_bytes - (size_t)(rest - (char*)ws), s));
  if (dmsg_time && d->d_time > 0) {
    const size_t esz = d->dtype == MTGNN_F32 ? 4 : 2;
    const void* Wt = (const char*)W_ih + esz * (size_t)(2 * dm);   // columns [2 dm, 2 dm + d_time)
    MTGNN_TRY(linear_dx(DP, dm, Wt, d->dtype, dmsg, dmsg_time, d->d_time, max_rows, n_rows, dm, d->d_time, false, s));
  }
  (void)W_hh;
  return MTGNN_OK;
}

// ---------------------------------------------------------------- time projection

mtgnn_status time_projection_impl(const int32_t* q_node, const float* q_t, const int32_t* n_q, int64_t max_q,
                                  const void* memory, const float* lu, const float* Wp, const float* bp, float scale,
                                  const mtgnn_dims* d, float* z, hipStream_t s) {
  if (max_q <= 0) return MTGNN_OK;
  const unsigned g = (unsigned)cdiv(max_q, 4);
  if (d->dtype == MTGNN_BF16)
    k_time_proj<uint16_t><<<g, 256, 0, s>>>(q_node, q_t, n_q, max_q, (const uint16_t*)memory, lu, Wp, bp, scale,
                                            d->d_mem, z);
  else
    k_time_proj<float><<<g, 256, 0, s>>>(q_node, q_t, n_q, max_q, (const float*)memory, lu, Wp, bp, scale, d->d_mem,
                                         z);
  MTGNN_CHECK_LAUNCH("time_proj");
  return MTGNN_OK;
}

struct ProjBwdWs {
  int32_t* row_of;
  uint32_t *keys, *vals;
  float *G, *Cq, *sums;
  void* sort_ws;
  size_t sort_bytes;
  void* cs_ws;
  size_t cs_bytes;
  void* seg_ws;      // the per-row sums of d M', for up to max_q updated rows
  size_t seg_bytes;
  size_t total;
};

static ProjBwdWs proj_bwd_layout(void* ws, const mtgnn_dims* d, int64_t max_q) {
  ProjBwdWs L{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    char* p = (char*)ws + off;
    off += a256j(bytes);
    return p;
  };
  const int64_t mq = max_q < 1 ? 1 : max_q;
  L.row_of = (int32_t*)take(sizeof(int32_t) * (size_t)d->n_nodes);
  L.keys = (uint32_t*)take(sizeof(uint32_t) * (size_t)mq);
  L.vals = (uint32_t*)take(sizeof(uint32_t) * (size_t)mq);
  L.G = (float*)take(sizeof(float) * (size_t)mq * 2 * d->d_mem);
  L.Cq = (float*)take(sizeof(float) * (size_t)mq * d->d_mem);
  L.sums = (float*)take(sizeof(float) * 2 * (size_t)d->d_mem);
  L.sort_bytes = radix_sort_ws_bytes(mq);
  L.sort_ws = take(L.sort_bytes);
  L.cs_bytes = colsum_ws_bytes(mq, 2 * d->d_mem);
  L.cs_ws = take(L.cs_bytes);
  L.seg_bytes = segsum_rows_ws_bytes(mq, mq, d->d_mem);
  L.seg_ws = take(L.seg_bytes);
  L.total = off;
  return L;
}

size_t time_projection_bwd_ws(const mtgnn_dims* d, int64_t max_q) {
  char base[1];
  return proj_bwd_layout(base, d, max_q).total;
}

mtgnn_status time_projection_bwd_impl(const int32_t* q_node, const float* q_t, const int32_t* n_q, int64_t max_q,
                                      const void* memory, const float* lu, const float* Wp, const float* bp,
                                      float scale, const float* dz, const int32_t* uniq, const int32_t* n_rows,
                                      int64_t max_rows, const mtgnn_dims* d, float* dWp, float* dbp, float* d_mem,
                                      void* ws, size_t ws_bytes, hipStream_t s) {
  if (ws_bytes < time_projection_bwd_ws(d, max_q)) return MTGNN_EWORKSPACE;
  ProjBwdWs L = proj_bwd_layout(ws, d, max_q);
  const int dm = d->d_mem;
  if (max_rows > 0) {
    k_jodie_row_map<<<(unsigned)cdiv(max_rows, 256), 256, 0, s>>>(uniq, n_rows, max_rows, L.row_of);
    MTGNN_CHECK_LAUNCH("jodie_row_map");
  }
  if (max_q > 0) {
    const unsigned g = (unsigned)cdiv(max_q, 4);
    if (d->dtype == MTGNN_BF16)
      k_time_proj_bwd_rows<uint16_t><<<g, 256, 0, s>>>(q_node, q_t, n_q, max_q, (const uint16_t*)memory, lu, scale, dm,
                                                       dz, uniq, n_rows, L.row_of, max_rows, Wp, bp, L.G, L.Cq, L.keys, L.vals);
    else
      k_time_proj_bwd_rows<float><<<g, 256, 0, s>>>(q_node, q_t, n_q, max_q, (const float*)memory, lu, scale, dm, dz,
                                                    uniq, n_rows, L.row_of, max_rows, Wp, bp, L.G, L.Cq, L.keys,
                                                    L.vals);
    MTGNN_CHECK_LAUNCH("time_proj_bwd_rows");
  }
  MTGNN_TRY(colsum(L.G, 2 * dm, max_q, n_q, 2 * dm, L.sums, false, L.cs_ws, L.cs_bytes, s));
  k_split_sums<<<(unsigned)cdiv(dm, 256), 256, 0, s>>>(L.sums, dm, dWp, dbp);
  MTGNN_CHECK_LAUNCH("split_sums");
  if (max_rows > 0) {
    uint32_t *sk = L.keys, *sv = L.vals;
    if (max_q > 0) MTGNN_TRY(radix_sort_pairs(&sk, &sv, max_q, bits_for(max_rows), L.sort_ws, L.sort_bytes, s));
    const unsigned g = (unsigned)cdiv(max_rows, 4);
    const bool lanes = dm % 4 == 0 && dm <= 128 && ((uintptr_t)L.Cq | (uintptr_t)d_mem) % 16 == 0;
    if (max_rows <= (max_q < 1 ? 1 : max_q) && dm <= 512)   // tiles of sorted occurrences, then the rows that span tiles
      MTGNN_TRY(segsum_rows(sk, sv, max_q, L.Cq, dm, dm, n_rows, max_rows, d_mem, L.seg_ws, L.seg_bytes, s));
    else if (lanes)
      k_jodie_dmem_lanes<32><<<g, 256, 0, s>>>(sk, sv, max_q, L.Cq, n_rows, max_rows, dm, d_mem);
    else if (d->dtype == MTGNN_BF16)
      k_jodie_dmem<uint16_t><<<g, 256, 0, s>>>(sk, sv, max_q, q_node, q_t, lu, Wp, bp, scale, dz, n_rows, max_rows, dm,
                                               d_mem);
    else
      k_jodie_dmem<float><<<g, 256, 0, s>>>(sk, sv, max_q, q_node, q_t, lu, Wp, bp, scale, dz, n_rows, max_rows, dm,
                                            d_mem);
    MTGNN_CHECK_LAUNCH("jodie_dmem");
  }
  return MTGNN_OK;
}

}  // namespace mtgnn

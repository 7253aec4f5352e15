// Temporal adjacency (built once per stream) and most-recent-k neighbour sampling.
#include "ops.h"

namespace mtgnn {

namespace {

size_t a256(size_t x) { return (x + 255) & ~size_t(255); }

// One wave per query: lower_bound of the query time in the node's time-sorted
// list by a 64-way search (each round the 64 lanes probe evenly spaced entries
// and the range shrinks 64-fold: a list of 4 M entries takes 4 dependent
// rounds), then the k entries just before it, newest first, one lane each.
__global__ __launch_bounds__(256) void k_sample_recent(const int64_t* __restrict__ off, const int32_t* __restrict__ nbr,
                                                       const float* __restrict__ t, const int32_t* __restrict__ eid,
                                                       const int32_t* __restrict__ q_node,
                                                       const float* __restrict__ q_t, const int32_t* __restrict__ n_q,
                                                       int64_t max_q, int k, int32_t* __restrict__ out_nbr,
                                                       float* __restrict__ out_t, int32_t* __restrict__ out_eid) {
  const int64_t q = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (q >= eff_count(max_q, n_q)) return;   // wave-uniform
  const int64_t n = q_node[q];
  const float tau = q_t[q];
  const int64_t lo = off[n];
  // invariant: the first entry with t >= tau lies in [a, b] (b: none)
  int64_t a = lo, b = off[n + 1];
  while (b - a > 64) {
    const int64_t step = (b - a + 63) >> 6;
    const int64_t p = a + (int64_t)(lane + 1) * step - 1;
    const bool lt = p < b && t[p] < tau;                       // true for a prefix of the lanes
    const int c = __popcll(__ballot(lt));
    const int64_t pc = a + (int64_t)(c + 1) * step - 1;        // probe of lane c: t >= tau there
    a += (int64_t)c * step;
    if (c < 64 && pc < b) b = pc;
  }
  const int64_t p = a + lane;
  const int64_t end = a + __popcll(__ballot(p < b && t[p] < tau));
  const int64_t o = q * k;
  for (int s = lane; s < k; s += 64) {
    const int64_t idx = end - 1 - s;
    if (idx >= lo) {
      out_nbr[o + s] = nbr[idx];
      out_t[o + s] = t[idx];
      out_eid[o + s] = eid[idx];
    } else {
      out_nbr[o + s] = -1;
      out_t[o + s] = 0.f;
      out_eid[o + s] = -1;
    }
  }
}

// Entry m = 2e + role belongs to node src[e] (role 0) or dst[e] (role 1).
__global__ void k_csr_keys(const int32_t* __restrict__ src, const int32_t* __restrict__ dst, int64_t n_events,
                           uint32_t* __restrict__ keys, uint32_t* __restrict__ vals) {
  const int64_t m = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (m >= 2 * n_events) return;
  const int64_t e = m >> 1;
  keys[m] = (uint32_t)((m & 1) ? dst[e] : src[e]);
  vals[m] = (uint32_t)m;
}

// off[n] = first sorted position whose node is >= n.
__global__ void k_csr_offsets(const uint32_t* __restrict__ keys, int64_t n_entries, int64_t n_nodes,
                              int64_t* __restrict__ off) {
  const int64_t n = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (n > n_nodes) return;
  int64_t a = 0, b = n_entries;
  while (a < b) {
    const int64_t mid = a + ((b - a) >> 1);
    if ((int64_t)keys[mid] < n) a = mid + 1;
    else b = mid;
  }
  off[n] = a;
}

__global__ void k_csr_fill(const uint32_t* __restrict__ vals, const int32_t* __restrict__ src,
                           const int32_t* __restrict__ dst, const float* __restrict__ t, int64_t n_entries,
                           int32_t* __restrict__ nbr, float* __restrict__ t_out, int32_t* __restrict__ eid_out) {
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= n_entries) return;
  const uint32_t m = vals[p];
  const int64_t e = m >> 1;
  nbr[p] = (m & 1) ? src[e] : dst[e];
  t_out[p] = t[e];
  eid_out[p] = (int32_t)e;
}

}  // namespace

mtgnn_status sample_recent_impl(const int64_t* off, const int32_t* nbr, const float* t, const int32_t* eid,
                                const int32_t* q_node, const float* q_t, const int32_t* n_q, int64_t max_q, int k,
                                int32_t* out_nbr, float* out_t, int32_t* out_eid, hipStream_t s) {
  if (max_q <= 0) return MTGNN_OK;
  k_sample_recent<<<(unsigned)cdiv(max_q, 4), 256, 0, s>>>(off, nbr, t, eid, q_node, q_t, n_q, max_q, k, out_nbr,
                                                            out_t, out_eid);
  MTGNN_CHECK_LAUNCH("sample_recent");
  return MTGNN_OK;
}

size_t build_csr_ws(int64_t n_events, int64_t) {
  const int64_t ne = 2 * n_events;
  return 2 * a256(sizeof(uint32_t) * ne) + radix_sort_ws_bytes(ne);
}

mtgnn_status build_csr_impl(const int32_t* src, const int32_t* dst, const float* t, int64_t n_events, int64_t n_nodes,
                            int64_t* off, int32_t* nbr, float* t_out, int32_t* eid_out, void* ws, size_t ws_bytes,
                            hipStream_t s) {
  const int64_t ne = 2 * n_events;
  if (ws_bytes < build_csr_ws(n_events, n_nodes)) return MTGNN_EWORKSPACE;
  char* w = (char*)ws;
  uint32_t* keys = (uint32_t*)w;
  w += a256(sizeof(uint32_t) * ne);
  uint32_t* vals = (uint32_t*)w;
  w += a256(sizeof(uint32_t) * ne);
  if (ne > 0) {
    k_csr_keys<<<(unsigned)cdiv(ne, 256), 256, 0, s>>>(src, dst, n_events, keys, vals);
    MTGNN_CHECK_LAUNCH("csr_keys");
    MTGNN_TRY(radix_sort_pairs(&keys, &vals, ne, bits_for(n_nodes - 1), w, ws_bytes - (size_t)(w - (char*)ws), s));
  }
  k_csr_offsets<<<(unsigned)cdiv(n_nodes + 1, 256), 256, 0, s>>>(keys, ne, n_nodes, off);
  MTGNN_CHECK_LAUNCH("csr_offsets");
  if (ne > 0) {
    k_csr_fill<<<(unsigned)cdiv(ne, 256), 256, 0, s>>>(vals, src, dst, t, ne, nbr, t_out, eid_out);
    MTGNN_CHECK_LAUNCH("csr_fill");
  }
  return MTGNN_OK;
}

}  // namespace mtgnn

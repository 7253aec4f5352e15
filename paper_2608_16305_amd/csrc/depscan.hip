// Offline backward dependency scan and mixed-batch construction (Algorithm 1, Section IV-B).
//
// One wave per (worker p, synchronization window q): the windows and the workers are independent
// scans, so a stream of W windows and P workers runs as P W waves.  A wave keeps its frontier F as a
// bitmap over the nodes (the candidate refresh set N_sync when the scan ends) and walks the window's
// batches latest first:
//   - the batch's target events (source owned by p) are marked, and their remote destinations join F;
//   - its other events are visited latest first, 64 at a time (lane 0 the latest): an event whose
//     source is remote and that touches F becomes an auxiliary replay event, and its remote
//     endpoints join F.  Within a chunk, lane l must see F as the earlier lanes' additions leave it:
//     the lanes that touch F as it stood at the chunk's start hit for certain; then the hit lanes are
//     taken in lane order, each one's remote endpoints broadcast, and any later lane that shares one
//     becomes a hit.  Lanes only ever activate later lanes, so this one sweep gives the sequential
//     result.
// F lives in global memory (it may exceed the LDS for large node counts); its reads are device-scope
// atomic loads and its updates atomic ORs, with a fence between a chunk's updates and the next reads.
#include "ops.h"

namespace mtgnn {

namespace {

__device__ __forceinline__ bool fbit(const uint32_t* F, int32_t x) {
  return (__hip_atomic_load(F + (x >> 5), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >> (x & 31)) & 1u;
}

__device__ __forceinline__ void fset(uint32_t* F, int32_t x) {
  __hip_atomic_fetch_or(F + (x >> 5), 1u << (x & 31), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__global__ __launch_bounds__(64) void k_dep_scan(const int32_t* __restrict__ src, const int32_t* __restrict__ dst,
                                                 int64_t E, const int32_t* __restrict__ owner, int n_workers,
                                                 int64_t batch, int window, int64_t n_windows, int64_t words,
                                                 uint8_t* __restrict__ role, uint32_t* __restrict__ sync) {
  const int64_t wq = blockIdx.x;
  const int p = (int)(wq / n_windows);
  const int64_t q = wq % n_windows;
  const int lane = threadIdx.x;
  const int64_t n_batches = cdiv(E, batch);
  const int64_t b_first = q * window;
  const int64_t b_last = min(n_batches, b_first + window) - 1;
  uint32_t* F = sync + wq * words;
  uint8_t* R = role + (int64_t)p * E;
  for (int64_t w = lane; w < words; w += 64) F[w] = 0u;
  for (int64_t e = b_first * batch + lane; e < min(E, (b_last + 1) * batch); e += 64) R[e] = 0;
  __threadfence();
  for (int64_t s = b_last; s >= b_first; --s) {
    const int64_t lo = s * batch, hi = min(E, lo + batch);
    // the batch's target events; their remote destinations join the frontier
    for (int64_t e = lo + lane; e < hi; e += 64) {
      if (owner[src[e]] == p) {
        R[e] = 1;
        const int32_t v = dst[e];
        if (owner[v] != p) fset(F, v);
      }
    }
    __threadfence();
    // the batch's other events, latest first
    for (int64_t c0 = hi - 1; c0 >= lo; c0 -= 64) {
      const int64_t e = c0 - lane;
      const bool valid = e >= lo;
      const int32_t u = valid ? src[e] : 0, v = valid ? dst[e] : 0;
      const bool cand = valid && owner[u] != p;
      const bool vrem = valid && owner[v] != p;
      bool me = cand && (fbit(F, u) || fbit(F, v));
      uint64_t hit = __ballot(me), done = 0;
      while (hit & ~done) {
        const int j = __ffsll((unsigned long long)(hit & ~done)) - 1;
        done |= 1ull << j;
        const int32_t uj = __shfl(u, j, 64), vj = __shfl(v, j, 64);
        const bool vjr = __shfl(vrem ? 1 : 0, j, 64) != 0;
        if (lane > j && cand && !me && (u == uj || v == uj || (vjr && (u == vj || v == vj)))) me = true;
        hit = __ballot(me);
      }
      if (me) {
        R[e] = 2;
        fset(F, u);
        if (vrem) fset(F, v);
      }
      __threadfence();
    }
  }
}

// mixed-batch compaction of one worker's roles
__global__ void k_role_ind(const uint8_t* __restrict__ role, int64_t E, int32_t* __restrict__ ind) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e < E) ind[e] = role[e] != 0 ? 1 : 0;
}

__global__ void k_role_scatter(const uint8_t* __restrict__ role, const int32_t* __restrict__ pos, int64_t E,
                               int64_t batch, int32_t* __restrict__ eid_out, uint8_t* __restrict__ flags_out,
                               int32_t* __restrict__ batch_off, const int32_t* __restrict__ total) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e < E) {
    const uint8_t r = role[e];
    if (r) {
      eid_out[pos[e]] = (int32_t)e;
      flags_out[pos[e]] = r == 2 ? 1 : 0;   // bit 0: auxiliary replay event
    }
    if (e % batch == 0) batch_off[e / batch] = pos[e];
  }
  if (e == 0) batch_off[cdiv(E, batch)] = *total;
}

size_t a256d(size_t x) { return (x + 255) & ~size_t(255); }

}  // namespace

mtgnn_status dep_scan_impl(const int32_t* src, const int32_t* dst, int64_t E, const int32_t* owner, int64_t n_nodes,
                           int n_workers, int64_t batch, int window, uint8_t* role, uint32_t* sync, hipStream_t s) {
  if (E <= 0) return MTGNN_OK;
  const int64_t n_windows = cdiv(cdiv(E, batch), window);
  const int64_t words = cdiv(n_nodes, 32);
  k_dep_scan<<<(unsigned)(n_workers * n_windows), 64, 0, s>>>(src, dst, E, owner, n_workers, batch, window, n_windows,
                                                              words, role, sync);
  MTGNN_CHECK_LAUNCH("dep_scan");
  return MTGNN_OK;
}

size_t mixed_batches_ws(int64_t E) { return 2 * a256d(sizeof(int32_t) * (size_t)(E < 1 ? 1 : E)) + 256 + scan_ws_bytes(E); }

mtgnn_status mixed_batches_impl(const uint8_t* role, int64_t E, int64_t batch, int32_t* eid_out, uint8_t* flags_out,
                                int32_t* batch_off, void* ws, size_t ws_bytes, hipStream_t s) {
  if (ws_bytes < mixed_batches_ws(E)) return MTGNN_EWORKSPACE;
  char* w = (char*)ws;
  int32_t* ind = (int32_t*)w;
  w += a256d(sizeof(int32_t) * (size_t)(E < 1 ? 1 : E));
  int32_t* pos = (int32_t*)w;
  w += a256d(sizeof(int32_t) * (size_t)(E < 1 ? 1 : E));
  int32_t* total = (int32_t*)w;
  w += 256;
  if (E <= 0) return MTGNN_OK;
  const unsigned g = (unsigned)cdiv(E, 256);
  k_role_ind<<<g, 256, 0, s>>>(role, E, ind);
  MTGNN_CHECK_LAUNCH("role_ind");
  MTGNN_TRY(scan_exclusive(ind, pos, E, total, w, ws_bytes - (size_t)(w - (char*)ws), s));
  k_role_scatter<<<g, 256, 0, s>>>(role, pos, E, batch, eid_out, flags_out, batch_off, total);
  MTGNN_CHECK_LAUNCH("role_scatter");
  return MTGNN_OK;
}

}  // namespace mtgnn

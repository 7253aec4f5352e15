// One-layer multi-head temporal attention embedding and its backward pass.
//
// Forward, per query q with k sampled neighbour slots:
//   q_in  = [M[q] || phi(0)]                 kv_in_j = [M[n_j] || x[e_j] || phi(tau - t_j)]
//   qv    = W_q q_in + b_q                   K_j, V_j = W_k kv_in_j + b_k, W_v kv_in_j + b_v
//   p     = softmax over valid j of qv_h . K_jh / sqrt(dh) per head h;  a_h = sum_j p_j V_jh
//   o     = W_o a + b_o;   z = W_2 relu(W_1 [o || M[q]] + b_1) + b_2
// The projections run on the MFMA GEMM; the gathers, per-query softmax and
// weighted sums are wave-per-query kernels.  Every intermediate the backward
// needs is kept in the save buffer.
#include "gemm.h"
#include "ops.h"

namespace mtgnn {

namespace {

size_t a256(size_t x) { return (x + 255) & ~size_t(255); }

struct AttnShape {
  int64_t Q, P;
  int dm, dt, de, da, H, dh, k, Dq, Dkv;
  explicit AttnShape(const mtgnn_dims* d, int64_t max_q) {
    Q = max_q; k = d->k; P = max_q * k;
    dm = d->d_mem; dt = d->d_time; de = d->d_edge; da = d->d_attn; H = d->n_heads; dh = da / H;
    Dq = dm + dt; Dkv = dm + de + dt;
  }
};

struct AttnSave {
  float *q_in, *kv_in, *qv, *KV, *p, *attn, *m_in, *m1, *a1;
  int32_t* npairs;
};

AttnSave carve_save(void* base, const AttnShape& s) {
  char* w = (char*)base;
  AttnSave v;
  auto take = [&](size_t bytes) { char* r = w; w += a256(bytes); return r; };
  v.q_in = (float*)take(sizeof(float) * s.Q * s.Dq);
  v.kv_in = (float*)take(sizeof(float) * s.P * s.Dkv);
  v.qv = (float*)take(sizeof(float) * s.Q * s.da);
  v.KV = (float*)take(sizeof(float) * s.P * 2 * s.da);
  v.p = (float*)take(sizeof(float) * s.Q * s.H * s.k);
  v.attn = (float*)take(sizeof(float) * s.Q * s.da);
  v.m_in = (float*)take(sizeof(float) * s.Q * (s.da + s.dm));
  v.m1 = (float*)take(sizeof(float) * s.Q * s.da);
  v.a1 = (float*)take(sizeof(float) * s.Q * s.da);
  v.npairs = (int32_t*)take(sizeof(int32_t));
  return v;
}

size_t save_total(const AttnShape& s) {
  return a256(sizeof(float) * s.Q * s.Dq) + a256(sizeof(float) * s.P * s.Dkv) + a256(sizeof(float) * s.Q * s.da) +
         a256(sizeof(float) * s.P * 2 * s.da) + a256(sizeof(float) * s.Q * s.H * s.k) +
         a256(sizeof(float) * s.Q * s.da) + a256(sizeof(float) * s.Q * (s.da + s.dm)) +
         2 * a256(sizeof(float) * s.Q * s.da) + a256(sizeof(int32_t));
}

__device__ __forceinline__ float pack_val(float v, int bf16) { return bf16 ? round_to_bf16(v) : v; }

__global__ void k_pairs_count(const int32_t* __restrict__ n_q, int64_t max_q, int k, int32_t* __restrict__ npairs) {
  const int64_t q = n_q ? (int64_t)(*n_q) : max_q;
  *npairs = (int32_t)((q < max_q ? q : max_q) * k);
}

template <typename T>
__global__ __launch_bounds__(256) void k_attn_gather_q(const int32_t* __restrict__ q_node,
                                                       const int32_t* __restrict__ n_q, int64_t max_q,
                                                       const T* __restrict__ mem, const float* __restrict__ tw,
                                                       const float* __restrict__ tb, int dm, int dt, int da, int bf16,
                                                       float* __restrict__ q_in, float* __restrict__ m_in) {
  const int64_t q = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (q >= eff_count(max_q, n_q)) return;
  const int64_t node = q_node[q];
  const int Dq = dm + dt;
  for (int c = lane; c < dm; c += 64) {
    const float v = Elem<T>::load(mem, node * dm + c);
    q_in[q * Dq + c] = v;
    m_in[q * (da + dm) + da + c] = v;
  }
  for (int j = lane; j < dt; j += 64) q_in[q * Dq + dm + j] = pack_val(cosf(time_arg(tw[j], 0.f, tb[j])), bf16);
}

template <typename T>
__global__ __launch_bounds__(256) void k_attn_gather_kv(const int32_t* __restrict__ nbr, const float* __restrict__ nt,
                                                        const int32_t* __restrict__ neid,
                                                        const float* __restrict__ q_t, const int32_t* __restrict__ n_q,
                                                        int64_t max_q, int k, const T* __restrict__ mem,
                                                        const float* __restrict__ x, const float* __restrict__ tw,
                                                        const float* __restrict__ tb, int dm, int de, int dt, int bf16,
                                                        float* __restrict__ kv_in) {
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int64_t q = r / k;
  if (q >= eff_count(max_q, n_q)) return;
  const int Dkv = dm + de + dt;
  float* row = kv_in + r * Dkv;
  const int64_t nb = nbr[r];
  if (nb < 0) {
    for (int c = lane; c < Dkv; c += 64) row[c] = 0.f;
    return;
  }
  for (int c = lane; c < dm; c += 64) row[c] = Elem<T>::load(mem, nb * dm + c);
  if (de > 0) {
    const float* xr = x + (int64_t)neid[r] * de;
    for (int c = lane; c < de; c += 64) row[dm + c] = pack_val(xr[c], bf16);
  }
  const float delta = q_t[q] - nt[r];
  for (int j = lane; j < dt; j += 64) row[dm + de + j] = pack_val(cosf(time_arg(tw[j], delta, tb[j])), bf16);
}

constexpr int MAX_DH_CHUNKS = 2;   // head width <= 128

// Wave per query: masked softmax over the k slots of each head, then the
// probability-weighted sum of the values.  Lane j < k holds slot j's score.
__global__ __launch_bounds__(256) void k_attn_core(const float* __restrict__ qv, const float* __restrict__ KV,
                                                   const int32_t* __restrict__ nbr, const int32_t* __restrict__ n_q,
                                                   int64_t max_q, int k, int da, int H, int bf16,
                                                   float* __restrict__ P, float* __restrict__ attn) {
  const int64_t q = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (q >= eff_count(max_q, n_q)) return;
  const int dh = da / H;
  const float scale = 1.0f / sqrtf((float)dh);
  for (int h = 0; h < H; ++h) {
    float qd[MAX_DH_CHUNKS];
#pragma unroll
    for (int c = 0; c < MAX_DH_CHUNKS; ++c) {
      const int d = lane + 64 * c;
      qd[c] = d < dh ? qv[q * da + h * dh + d] : 0.f;
    }
    float my_s = -INFINITY;
    for (int j = 0; j < k; ++j) {
      const int64_t r = q * k + j;
      float part = 0.f;
#pragma unroll
      for (int c = 0; c < MAX_DH_CHUNKS; ++c) {
        const int d = lane + 64 * c;
        if (d < dh) part += qd[c] * KV[r * 2 * da + h * dh + d];
      }
      const float s = wave_sum(part) * scale;
      if (lane == j) my_s = nbr[r] >= 0 ? s : -INFINITY;
    }
    const float m = wave_max(my_s);
    const float e = (lane < k && my_s > -INFINITY) ? expf(my_s - m) : 0.f;
    const float den = wave_sum(e);
    const float pj = den > 0.f ? e / den : 0.f;
    if (lane < k) P[(q * H + h) * k + lane] = pj;
    float acc[MAX_DH_CHUNKS] = {0.f, 0.f};
    for (int j = 0; j < k; ++j) {
      const float pb = __shfl(pj, j, 64);
      const int64_t r = q * k + j;
#pragma unroll
      for (int c = 0; c < MAX_DH_CHUNKS; ++c) {
        const int d = lane + 64 * c;
        if (d < dh) acc[c] += pb * KV[r * 2 * da + da + h * dh + d];
      }
    }
#pragma unroll
    for (int c = 0; c < MAX_DH_CHUNKS; ++c) {
      const int d = lane + 64 * c;
      if (d < dh) attn[q * da + h * dh + d] = pack_val(acc[c], bf16);
    }
  }
}

// Wave per query: gradients of the softmax-weighted sum and of the scores.
//   dV_j = p_j da_h;  dp_j = da_h . V_j;  ds_j = p_j (dp_j - sum_i p_i dp_i)
//   dq_h = sum_j ds_j K_jh / sqrt(dh);  dK_j = ds_j q_h / sqrt(dh)
__global__ __launch_bounds__(256) void k_attn_core_bwd(const float* __restrict__ qv, const float* __restrict__ KV,
                                                       const float* __restrict__ P, const float* __restrict__ dattn,
                                                       const int32_t* __restrict__ n_q, int64_t max_q, int k, int da,
                                                       int H, float* __restrict__ dKV, float* __restrict__ dqv) {
  const int64_t q = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (q >= eff_count(max_q, n_q)) return;
  const int dh = da / H;
  const float scale = 1.0f / sqrtf((float)dh);
  for (int h = 0; h < H; ++h) {
    float qd[MAX_DH_CHUNKS], gd[MAX_DH_CHUNKS];
#pragma unroll
    for (int c = 0; c < MAX_DH_CHUNKS; ++c) {
      const int d = lane + 64 * c;
      qd[c] = d < dh ? qv[q * da + h * dh + d] : 0.f;
      gd[c] = d < dh ? dattn[q * da + h * dh + d] : 0.f;
    }
    const float pl = lane < k ? P[(q * H + h) * k + lane] : 0.f;
    float my_dp = 0.f;
    for (int j = 0; j < k; ++j) {
      const int64_t r = q * k + j;
      float part = 0.f;
#pragma unroll
      for (int c = 0; c < MAX_DH_CHUNKS; ++c) {
        const int d = lane + 64 * c;
        if (d < dh) part += gd[c] * KV[r * 2 * da + da + h * dh + d];
      }
      const float dp = wave_sum(part);
      if (lane == j) my_dp = dp;
    }
    const float sdp = wave_sum(pl * my_dp);
    const float dsl = pl * (my_dp - sdp);
    float dq[MAX_DH_CHUNKS] = {0.f, 0.f};
    for (int j = 0; j < k; ++j) {
      const float dsj = __shfl(dsl, j, 64);
      const float pj = __shfl(pl, j, 64);
      const int64_t r = q * k + j;
#pragma unroll
      for (int c = 0; c < MAX_DH_CHUNKS; ++c) {
        const int d = lane + 64 * c;
        if (d < dh) {
          dq[c] += dsj * KV[r * 2 * da + h * dh + d];
          dKV[r * 2 * da + h * dh + d] = dsj * qd[c] * scale;
          dKV[r * 2 * da + da + h * dh + d] = pj * gd[c];
        }
      }
    }
#pragma unroll
    for (int c = 0; c < MAX_DH_CHUNKS; ++c) {
      const int d = lane + 64 * c;
      if (d < dh) dqv[q * da + h * dh + d] = dq[c] * scale;
    }
  }
}

// ---------------------------------------------------------------- d M' by node (deterministic)

// Occurrence o < Q is query o, o >= Q is neighbour slot o - Q.  Its key is the
// row of its node in `uniq` (ascending), or `sentinel` when the node was not
// updated this step, the slot is empty or the query is beyond n_q.
__global__ void k_occ_keys(const int32_t* __restrict__ q_node, const int32_t* __restrict__ nbr,
                           const int32_t* __restrict__ n_q, int64_t max_q, int k, const int32_t* __restrict__ uniq,
                           const int32_t* __restrict__ n_rows, int64_t max_rows, uint32_t sentinel,
                           uint32_t* __restrict__ keys, uint32_t* __restrict__ vals) {
  const int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t n_occ = max_q * (1 + k);
  if (o >= n_occ) return;
  const int64_t nq = eff_count(max_q, n_q);
  int64_t node = -1;
  if (o < max_q) {
    if (o < nq) node = q_node[o];
  } else {
    const int64_t r = o - max_q;
    if (r / k < nq) node = nbr[r];
  }
  uint32_t key = sentinel;
  if (node >= 0) {
    const int64_t nr = eff_count(max_rows, n_rows);
    int64_t a = 0, b = nr;
    while (a < b) {
      const int64_t mid = a + ((b - a) >> 1);
      if ((int64_t)uniq[mid] < node) a = mid + 1;
      else b = mid;
    }
    if (a < nr && uniq[a] == node) key = (uint32_t)a;
  }
  keys[o] = key;
  vals[o] = (uint32_t)o;
}

constexpr int SEG_TILE = 64;     // sorted occurrences per wave
constexpr int SEG_MAXC = 8;      // columns per lane: width <= 512

struct SegCtx {
  const uint32_t* keys;
  const uint32_t* vals;
  int64_t n_occ;
  uint32_t sentinel;
  int64_t max_q;
  const float* dhq;   // [Q, ldq] query-side gradient of M[q] (columns [0, dm))
  int64_t ldq;
  const float* dkv;   // [P, 2 da] neighbour-slot gradient of (K, V)
  int dm, w2;         // w2 = 2 da ; row width W = dm + w2
  float* S;           // [rows, W] complete sums
  float* head;        // [ntiles, W]
  float* tail;        // [ntiles, W]
};

__device__ __forceinline__ void seg_add(const SegCtx& c, uint32_t o, float* acc, int lane) {
  const int W = c.dm + c.w2;
  if ((int64_t)o < c.max_q) {
    const float* src = c.dhq + (int64_t)o * c.ldq;
#pragma unroll
    for (int i = 0; i < SEG_MAXC; ++i) {
      const int col = lane + 64 * i;
      if (col < c.dm) acc[i] += src[col];
    }
  } else {
    const float* src = c.dkv + ((int64_t)o - c.max_q) * c.w2;
#pragma unroll
    for (int i = 0; i < SEG_MAXC; ++i) {
      const int col = lane + 64 * i;
      if (col >= c.dm && col < W) acc[i] += src[col - c.dm];
    }
  }
}

__device__ __forceinline__ void seg_store(float* dst, const float* acc, int W, int lane) {
#pragma unroll
  for (int i = 0; i < SEG_MAXC; ++i) {
    const int col = lane + 64 * i;
    if (col < W) dst[col] = acc[i];
  }
}

// Wave per tile of SEG_TILE sorted positions.  A segment (one row) entirely
// inside the tile is written to S; the piece of a segment that began before
// the tile goes to head[tile]; the piece of one that continues past it goes
// to tail[tile].  The fixup pass adds the pieces in tile order.
__global__ __launch_bounds__(256) void k_segsum_tiles(SegCtx c) {
  const int64_t tile = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int64_t p0 = tile * SEG_TILE;
  if (p0 >= c.n_occ) return;
  const int64_t p1 = min(c.n_occ, p0 + SEG_TILE);
  const int W = c.dm + c.w2;
  uint32_t cur = c.keys[p0];
  if (cur == c.sentinel) return;
  float acc[SEG_MAXC];
#pragma unroll
  for (int i = 0; i < SEG_MAXC; ++i) acc[i] = 0.f;
  bool first = true;
  int64_t p = p0;
  for (; p < p1; ++p) {
    const uint32_t key = c.keys[p];
    if (key != cur) {
      const bool before = first && p0 > 0 && c.keys[p0 - 1] == cur;
      seg_store(before ? c.head + tile * W : c.S + (int64_t)cur * W, acc, W, lane);
#pragma unroll
      for (int i = 0; i < SEG_MAXC; ++i) acc[i] = 0.f;
      first = false;
      cur = key;
      if (key == c.sentinel) break;
    }
    seg_add(c, c.vals[p], acc, lane);
  }
  if (p == p1) {   // the last piece reached the tile end
    const bool before = first && p0 > 0 && c.keys[p0 - 1] == cur;
    const bool after = p1 < c.n_occ && c.keys[p1] == cur;
    float* dst = before ? c.head + tile * W : (after ? c.tail + tile * W : c.S + (int64_t)cur * W);
    seg_store(dst, acc, W, lane);
  }
}

__device__ __forceinline__ int64_t lower_bound_u32(const uint32_t* a, int64_t n, uint32_t v) {
  int64_t lo = 0, hi = n;
  while (lo < hi) {
    const int64_t mid = lo + ((hi - lo) >> 1);
    if (a[mid] < v) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

__global__ __launch_bounds__(256) void k_segsum_fixup(SegCtx c, const int32_t* __restrict__ n_rows,
                                                      int64_t max_rows) {
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= eff_count(max_rows, n_rows)) return;
  const int W = c.dm + c.w2;
  const int64_t a = lower_bound_u32(c.keys, c.n_occ, (uint32_t)r);
  const int64_t b = lower_bound_u32(c.keys, c.n_occ, (uint32_t)r + 1);
  float acc[SEG_MAXC];
#pragma unroll
  for (int i = 0; i < SEG_MAXC; ++i) acc[i] = 0.f;
  if (a < b) {
    const int64_t t0 = a / SEG_TILE, t1 = (b - 1) / SEG_TILE;
    if (t0 == t1) return;   // written whole by its tile
    const float* src = c.tail + t0 * W;
#pragma unroll
    for (int i = 0; i < SEG_MAXC; ++i) {
      const int col = lane + 64 * i;
      if (col < W) acc[i] = src[col];
    }
    for (int64_t t = t0 + 1; t <= t1; ++t) {
      src = c.head + t * W;
#pragma unroll
      for (int i = 0; i < SEG_MAXC; ++i) {
        const int col = lane + 64 * i;
        if (col < W) acc[i] += src[col];
      }
    }
  }
  seg_store(c.S + r * W, acc, W, lane);
}

__global__ void k_copy_cols(const float* __restrict__ S, int64_t lds, const int32_t* __restrict__ n_rows,
                            int64_t max_rows, int cols, float* __restrict__ out, int64_t ldo) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t r = e / cols;
  if (r >= eff_count(max_rows, n_rows)) return;
  const int c = (int)(e % cols);
  out[r * ldo + c] = S[r * lds + c];
}

struct BwdWs {
  float *dm1, *dm_in, *dattn, *dqv, *dphi0, *dKV, *dphin, *S, *head, *tail;
  uint32_t *keys, *vals;
  char* scratch;
  size_t scratch_bytes;
  size_t total;
};

BwdWs carve_bwd(void* base, const AttnShape& s, int64_t max_rows) {
  char* w = (char*)base;
  BwdWs v;
  auto take = [&](size_t bytes) { char* r = w; w += a256(bytes); return r; };
  const int64_t n_occ = s.Q * (1 + s.k);
  const int64_t ntiles = cdiv(n_occ, SEG_TILE);
  const int W = s.dm + 2 * s.da;
  v.dm1 = (float*)take(sizeof(float) * s.Q * s.da);
  v.dm_in = (float*)take(sizeof(float) * s.Q * (s.da + s.dm));
  v.dattn = (float*)take(sizeof(float) * s.Q * s.da);
  v.dqv = (float*)take(sizeof(float) * s.Q * s.da);
  v.dphi0 = (float*)take(sizeof(float) * s.Q * (s.dt > 0 ? s.dt : 1));
  v.dKV = (float*)take(sizeof(float) * s.P * 2 * s.da);
  v.dphin = (float*)take(sizeof(float) * s.P * (s.dt > 0 ? s.dt : 1));
  v.S = (float*)take(sizeof(float) * (max_rows > 0 ? max_rows : 1) * W);
  v.head = (float*)take(sizeof(float) * ntiles * W);
  v.tail = (float*)take(sizeof(float) * ntiles * W);
  v.keys = (uint32_t*)take(sizeof(uint32_t) * n_occ);
  v.vals = (uint32_t*)take(sizeof(uint32_t) * n_occ);
  size_t sc = radix_sort_ws_bytes(n_occ);
  auto mx = [&](size_t x) { if (x > sc) sc = x; };
  mx(linear_dw_ws_bytes(s.Q, s.da, s.da + s.dm));
  mx(linear_dw_ws_bytes(s.Q, s.da, s.Dq));
  mx(linear_dw_ws_bytes(s.P, s.da, s.Dkv));
  mx(colsum_ws_bytes(s.P, s.da));
  mx(colsum_ws_bytes(s.Q, s.da));
  mx(timegrad_ws_bytes(s.P, s.dt));
  mx(timegrad_ws_bytes(s.Q, s.dt));
  v.scratch = take(sc);
  v.scratch_bytes = a256(sc);
  v.total = (size_t)(w - (char*)base);
  return v;
}

}  // namespace

size_t attn_save_bytes(const mtgnn_dims* d, int64_t max_q) { return save_total(AttnShape(d, max_q)); }

size_t attn_fwd_ws(const mtgnn_dims*, int64_t) { return 0; }

mtgnn_status attn_fwd_impl(const int32_t* q_node, const float* q_t, const int32_t* n_q, int64_t max_q,
                           const int32_t* nbr, const float* nt, const int32_t* neid, const void* memory,
                           const float* edge_feat, const float* tw, const float* tb, const mtgnn_attn_params* p,
                           const mtgnn_dims* d, float* z, void* save, void*, size_t, hipStream_t s) {
  const AttnShape sh(d, max_q);
  const AttnSave sv = carve_save(save, sh);
  const int bf = d->dtype == MTGNN_BF16 ? 1 : 0;
  const int wt = d->dtype;
  k_pairs_count<<<1, 1, 0, s>>>(n_q, max_q, sh.k, sv.npairs);
  MTGNN_CHECK_LAUNCH("pairs_count");
  const unsigned gq = (unsigned)cdiv(sh.Q, 4), gp = (unsigned)cdiv(sh.P, 4);
  if (!bf) {
    k_attn_gather_q<float><<<gq, 256, 0, s>>>(q_node, n_q, max_q, (const float*)memory, tw, tb, sh.dm, sh.dt, sh.da, 0,
                                              sv.q_in, sv.m_in);
    k_attn_gather_kv<float><<<gp, 256, 0, s>>>(nbr, nt, neid, q_t, n_q, max_q, sh.k, (const float*)memory, edge_feat,
                                               tw, tb, sh.dm, sh.de, sh.dt, 0, sv.kv_in);
  } else {
    k_attn_gather_q<uint16_t><<<gq, 256, 0, s>>>(q_node, n_q, max_q, (const uint16_t*)memory, tw, tb, sh.dm, sh.dt,
                                                 sh.da, 1, sv.q_in, sv.m_in);
    k_attn_gather_kv<uint16_t><<<gp, 256, 0, s>>>(nbr, nt, neid, q_t, n_q, max_q, sh.k, (const uint16_t*)memory,
                                                  edge_feat, tw, tb, sh.dm, sh.de, sh.dt, 1, sv.kv_in);
  }
  MTGNN_CHECK_LAUNCH("attn_gather");
  MTGNN_TRY(linear_fwd(sv.q_in, MTGNN_F32, sh.Dq, p->W_q, wt, sh.Dq, p->b_q, sv.qv, sh.da, sh.Q, n_q, sh.da, sh.Dq,
                       false, s));
  MTGNN_TRY(linear_fwd(sv.kv_in, MTGNN_F32, sh.Dkv, p->W_k, wt, sh.Dkv, p->b_k, sv.KV, 2 * sh.da, sh.P, sv.npairs,
                       sh.da, sh.Dkv, false, s));
  MTGNN_TRY(linear_fwd(sv.kv_in, MTGNN_F32, sh.Dkv, p->W_v, wt, sh.Dkv, p->b_v, sv.KV + sh.da, 2 * sh.da, sh.P,
                       sv.npairs, sh.da, sh.Dkv, false, s));
  k_attn_core<<<gq, 256, 0, s>>>(sv.qv, sv.KV, nbr, n_q, max_q, sh.k, sh.da, sh.H, bf, sv.p, sv.attn);
  MTGNN_CHECK_LAUNCH("attn_core");
  const int64_t ldm = sh.da + sh.dm;
  MTGNN_TRY(linear_fwd(sv.attn, MTGNN_F32, sh.da, p->W_o, wt, sh.da, p->b_o, sv.m_in, ldm, sh.Q, n_q, sh.da, sh.da,
                       false, s, nullptr, 0, bf != 0));
  MTGNN_TRY(linear_fwd(sv.m_in, MTGNN_F32, ldm, p->W_1, wt, ldm, p->b_1, sv.a1, sh.da, sh.Q, n_q, sh.da, ldm, false, s,
                       sv.m1, sh.da, bf != 0));
  MTGNN_TRY(linear_fwd(sv.a1, MTGNN_F32, sh.da, p->W_2, wt, sh.da, p->b_2, z, sh.da, sh.Q, n_q, sh.da, sh.da, false,
                       s));
  return MTGNN_OK;
}

size_t attn_bwd_ws(const mtgnn_dims* d, int64_t max_q, int64_t max_rows) {
  return carve_bwd(nullptr, AttnShape(d, max_q), max_rows).total;
}

mtgnn_status attn_bwd_impl(const int32_t* q_node, const float* q_t, const int32_t* n_q, int64_t max_q,
                           const int32_t* nbr, const float* nt, const float* dz, const void* save, const int32_t* uniq,
                           const int32_t* n_rows, int64_t max_rows, const float* tw, const float* tb,
                           const mtgnn_attn_params* p, const mtgnn_dims* d, mtgnn_attn_grads* g, float* d_mem,
                           float* d_time_w, float* d_time_b, void* ws, size_t ws_bytes, hipStream_t s) {
  const AttnShape sh(d, max_q);
  const AttnSave sv = carve_save((void*)save, sh);
  const BwdWs b = carve_bwd(ws, sh, max_rows);
  if (ws_bytes < b.total) return MTGNN_EWORKSPACE;
  const int wt = d->dtype;
  const size_t esz = wt == MTGNN_F32 ? 4 : 2;
  const int64_t Q = sh.Q, P = sh.P, ldm = sh.da + sh.dm;
  const int da = sh.da, dm = sh.dm, dt = sh.dt;
  char* sc = b.scratch;
  const size_t scb = b.scratch_bytes;
  auto wofs = [&](const void* W, int64_t col) { return (const void*)((const char*)W + esz * (size_t)col); };

  // merge MLP: z = W_2 a1 + b_2, a1 = relu(m1), m1 = W_1 m_in + b_1
  MTGNN_TRY(linear_dw(dz, da, sv.a1, MTGNN_F32, da, g->W_2, da, Q, n_q, da, da, sc, scb, s));
  MTGNN_TRY(colsum(dz, da, Q, n_q, da, g->b_2, false, sc, scb, s));
  MTGNN_TRY(linear_dx(dz, da, p->W_2, wt, da, b.dm1, da, Q, n_q, da, da, false, s, sv.m1, da));
  MTGNN_TRY(linear_dw(b.dm1, da, sv.m_in, MTGNN_F32, ldm, g->W_1, ldm, Q, n_q, da, ldm, sc, scb, s));
  MTGNN_TRY(colsum(b.dm1, da, Q, n_q, da, g->b_1, false, sc, scb, s));
  MTGNN_TRY(linear_dx(b.dm1, da, p->W_1, wt, ldm, b.dm_in, ldm, Q, n_q, da, ldm, false, s));
  // output projection: o = W_o attn + b_o   (do = dm_in[:, :da])
  MTGNN_TRY(linear_dw(b.dm_in, ldm, sv.attn, MTGNN_F32, da, g->W_o, da, Q, n_q, da, da, sc, scb, s));
  MTGNN_TRY(colsum(b.dm_in, ldm, Q, n_q, da, g->b_o, false, sc, scb, s));
  MTGNN_TRY(linear_dx(b.dm_in, ldm, p->W_o, wt, da, b.dattn, da, Q, n_q, da, da, false, s));
  // softmax-weighted sum and scores
  k_attn_core_bwd<<<(unsigned)cdiv(Q, 4), 256, 0, s>>>(sv.qv, sv.KV, sv.p, b.dattn, n_q, max_q, sh.k, da, sh.H, b.dKV,
                                                        b.dqv);
  MTGNN_CHECK_LAUNCH("attn_core_bwd");
  // query projection: dhq += dqv W_q[:, :dm];  dphi(0) = dqv W_q[:, dm:]
  MTGNN_TRY(linear_dw(b.dqv, da, sv.q_in, MTGNN_F32, sh.Dq, g->W_q, sh.Dq, Q, n_q, da, sh.Dq, sc, scb, s));
  MTGNN_TRY(colsum(b.dqv, da, Q, n_q, da, g->b_q, false, sc, scb, s));
  MTGNN_TRY(linear_dx(b.dqv, da, p->W_q, wt, sh.Dq, b.dm_in + da, ldm, Q, n_q, da, dm, true, s));
  if (dt > 0) {
    MTGNN_TRY(linear_dx(b.dqv, da, wofs(p->W_q, dm), wt, sh.Dq, b.dphi0, dt, Q, n_q, da, dt, false, s));
    MTGNN_TRY(timegrad_zero(b.dphi0, dt, Q, n_q, tw, tb, dt, d_time_w, d_time_b, false, sc, scb, s));
  }
  // key/value projections over the neighbour slots
  MTGNN_TRY(linear_dw(b.dKV, 2 * da, sv.kv_in, MTGNN_F32, sh.Dkv, g->W_k, sh.Dkv, P, sv.npairs, da, sh.Dkv, sc, scb,
                      s));
  MTGNN_TRY(linear_dw(b.dKV + da, 2 * da, sv.kv_in, MTGNN_F32, sh.Dkv, g->W_v, sh.Dkv, P, sv.npairs, da, sh.Dkv, sc,
                      scb, s));
  MTGNN_TRY(colsum(b.dKV, 2 * da, P, sv.npairs, da, g->b_k, false, sc, scb, s));
  MTGNN_TRY(colsum(b.dKV + da, 2 * da, P, sv.npairs, da, g->b_v, false, sc, scb, s));
  if (dt > 0) {
    const int64_t tcol = dm + sh.de;
    MTGNN_TRY(linear_dx(b.dKV, 2 * da, wofs(p->W_k, tcol), wt, sh.Dkv, b.dphin, dt, P, sv.npairs, da, dt, false, s));
    MTGNN_TRY(linear_dx(b.dKV + da, 2 * da, wofs(p->W_v, tcol), wt, sh.Dkv, b.dphin, dt, P, sv.npairs, da, dt, true,
                        s));
    MTGNN_TRY(timegrad_pairs(b.dphin, dt, P, n_q, sh.k, nbr, q_t, nt, tw, tb, dt, d_time_w, d_time_b, true, sc, scb,
                             s));
  }
  // d M' for the updated rows: group every occurrence by row, sum in a fixed order
  if (max_rows > 0) {
    const int64_t n_occ = Q * (1 + sh.k);
    const uint32_t sentinel = (uint32_t)max_rows;
    k_occ_keys<<<(unsigned)cdiv(n_occ, 256), 256, 0, s>>>(q_node, nbr, n_q, max_q, sh.k, uniq, n_rows, max_rows,
                                                           sentinel, b.keys, b.vals);
    MTGNN_CHECK_LAUNCH("occ_keys");
    MTGNN_TRY(radix_sort_pairs(b.keys, b.vals, n_occ, bits_for(max_rows), sc, scb, s));
    SegCtx c;
    c.keys = b.keys; c.vals = b.vals; c.n_occ = n_occ; c.sentinel = sentinel; c.max_q = max_q;
    c.dhq = b.dm_in + da; c.ldq = ldm; c.dkv = b.dKV; c.dm = dm; c.w2 = 2 * da;
    c.S = b.S; c.head = b.head; c.tail = b.tail;
    const int64_t ntiles = cdiv(n_occ, SEG_TILE);
    k_segsum_tiles<<<(unsigned)cdiv(ntiles, 4), 256, 0, s>>>(c);
    MTGNN_CHECK_LAUNCH("segsum_tiles");
    k_segsum_fixup<<<(unsigned)cdiv(max_rows, 4), 256, 0, s>>>(c, n_rows, max_rows);
    MTGNN_CHECK_LAUNCH("segsum_fixup");
    const int W = dm + 2 * da;
    k_copy_cols<<<(unsigned)cdiv(max_rows * dm, 256), 256, 0, s>>>(b.S, W, n_rows, max_rows, dm, d_mem, dm);
    MTGNN_CHECK_LAUNCH("copy_cols");
    MTGNN_TRY(linear_dx(b.S + dm, W, p->W_k, wt, sh.Dkv, d_mem, dm, max_rows, n_rows, da, dm, true, s));
    MTGNN_TRY(linear_dx(b.S + dm + da, W, p->W_v, wt, sh.Dkv, d_mem, dm, max_rows, n_rows, da, dm, true, s));
  }
  return MTGNN_OK;
}

}  // namespace mtgnn

// One-layer multi-head temporal attention embedding and its backward pass.
//
// Forward, per query q with k sampled neighbour slots:
//   q_in  = [M[q] || phi(0)]                 kv_in_j = [M[n_j] || x[e_j] || phi(tau - t_j)]
//   qv    = W_q q_in + b_q                   [K_j | V_j] = [W_k; W_v] kv_in_j + [b_k; b_v]
//   p     = softmax over valid j of qv_h . K_jh / sqrt(dh) per head h;  a_h = sum_j p_j V_jh
//   o     = W_o a + b_o;   z = W_2 relu(W_1 [o || M[q]] + b_1) + b_2
//
// Neighbour slots are compacted: sampling pads each query's slots at the
// tail, so the valid slots of query q are j < cnt[q], stored at rows
// pair_off[q] + j of every per-slot array (kv_in, K|V, their gradients).  The
// key/value projection, its weight gradient and its data gradient therefore
// run only over real neighbours.  K and V share one product against the
// stacked weights [W_k; W_v] (kept in the save buffer for the backward).
// The projections run on the MFMA strip GEMM; gathers, per-query softmax and
// weighted sums are wave-per-query kernels.
#include "gemm.h"
#include "ops.h"

namespace mtgnn {

namespace {

size_t a256(size_t x) { return (x + 255) & ~size_t(255); }

struct AttnShape {
  int64_t Q, P, N;
  int dm, dt, de, da, H, dh, k, Dq, Dkv;
  size_t esz;   // bytes per weight element
  explicit AttnShape(const mtgnn_dims* d, int64_t max_q) {
    Q = max_q; k = d->k; P = max_q * k; N = d->n_nodes;
    dm = d->d_mem; dt = d->d_time; de = d->d_edge; da = d->d_attn; H = d->n_heads; dh = da / H;
    Dq = dm + dt; Dkv = dm + de + dt;
    esz = d->dtype == MTGNN_F32 ? 4 : 2;
  }
};

// Save buffer: written by the forward, read by the backward.
struct AttnSave {
  void* W_kv;            // [2 da, Dkv] stacked [W_k; W_v] (weight dtype)
  float* b_kv;           // [2 da]
  int32_t *cnt, *pair_off, *n_valid, *pair_nbr;
  float *pair_delta;     // per compact slot: tau - t_j
  float *q_in, *kv_in, *qv, *KV, *p, *attn, *m_in, *m1, *a1;
  float* merge_w;        // zero-padded merge weights and their transposes for the fused chains (float32 only)
  float* qc;             // the query projection's constant b_q + W_q[:, dm:] phi(0) (fused float32 path)
  size_t total;
};

AttnSave carve_save(void* base, const AttnShape& s) {
  char* w = (char*)base;
  AttnSave v;
  auto take = [&](size_t bytes) { char* r = w; w += a256(bytes); return r; };
  // the weight copies first: their offsets do not depend on the query count (the weights-only
  // preparation carves with none)
  v.W_kv = take(s.esz * 2 * s.da * s.Dkv);
  v.b_kv = (float*)take(sizeof(float) * 2 * s.da);
  v.merge_w = (float*)take(sizeof(float) * (s.esz == 4 ? merge_weights_floats(s.da, s.dm, s.dt) : 1));
  v.qc = (float*)take(sizeof(float) * s.da);
  v.cnt = (int32_t*)take(sizeof(int32_t) * s.Q);
  v.pair_off = (int32_t*)take(sizeof(int32_t) * s.Q);
  v.n_valid = (int32_t*)take(sizeof(int32_t));
  v.pair_nbr = (int32_t*)take(sizeof(int32_t) * s.P);
  v.pair_delta = (float*)take(sizeof(float) * s.P);
  v.q_in = (float*)take(sizeof(float) * s.Q * s.Dq);
  v.kv_in = (float*)take(sizeof(float) * s.P * s.Dkv);
  v.qv = (float*)take(sizeof(float) * s.Q * s.da);
  v.KV = (float*)take(sizeof(float) * s.P * 2 * s.da);
  v.p = (float*)take(sizeof(float) * s.Q * s.H * s.k);
  v.attn = (float*)take(sizeof(float) * s.Q * s.da);
  v.m_in = (float*)take(sizeof(float) * s.Q * (s.da + s.dm));
  v.m1 = (float*)take(sizeof(float) * s.Q * s.da);
  v.a1 = (float*)take(sizeof(float) * s.Q * s.da);
  v.total = (size_t)(w - (char*)base);
  return v;
}

__device__ __forceinline__ float pack_val(float v, int bf16) { return bf16 ? round_to_bf16(v) : v; }

// Stack [W_k; W_v] and [b_k; b_v] (a few hundred KB; once per forward).
template <typename T>
__global__ void k_stack_kv(const T* __restrict__ Wk, const T* __restrict__ Wv, const float* __restrict__ bk,
                           const float* __restrict__ bv, int da, int Dkv, T* __restrict__ W, float* __restrict__ b) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t half = (int64_t)da * Dkv;
  if (e < half) {
    W[e] = Wk[e];
    W[half + e] = Wv[e];
  }
  if (e < da) {
    b[e] = bk[e];
    b[da + e] = bv[e];
  }
}

// cnt[q] = number of valid (leading) slots; 0 beyond the device query count.
__global__ void k_pair_counts(const int32_t* __restrict__ nbr, const int32_t* __restrict__ n_q, int64_t max_q, int k,
                              int32_t* __restrict__ cnt) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= max_q) return;
  int c = 0;
  if (q < eff_count(max_q, n_q))
    while (c < k && nbr[q * k + c] >= 0) ++c;
  cnt[q] = c;
}

template <typename T>
__device__ __forceinline__ void gather_q_body(int64_t q, int lane, const int32_t* __restrict__ q_node,
                                              const T* __restrict__ mem, const float* __restrict__ tw,
                                              const float* __restrict__ tb, int dm, int dt, int da, int bf16,
                                              float* __restrict__ q_in, float* __restrict__ m_in) {
  const int64_t node = q_node[q];
  const int Dq = dm + dt;
  for (int c = lane; c < dm; c += 64) {
    const float v = Elem<T>::load(mem, node * dm + c);
    q_in[q * Dq + c] = v;
    m_in[q * (da + dm) + da + c] = v;
  }
  for (int j = lane; j < dt; j += 64) {
    const float arg = time_arg(tw[j], 0.f, tb[j]);
    q_in[q * Dq + dm + j] = bf16 ? round_to_bf16(cos_for_bf16(arg)) : cosf(arg);
  }
}

// Wave per query: the rows of its valid slots, [M[n_j] || x[e_j] || cos(w (tau - t_j) + b)],
// the slot's node and its tau - t_j.
// Slots go GATHER_CHUNK at a time: the chunk's memory-row loads are all issued before any is stored.
constexpr int GATHER_CHUNK = 8;

template <typename T>
__device__ __forceinline__ void gather_kv_body(int64_t q, int lane, const int32_t* __restrict__ nbr,
                                               const float* __restrict__ nt, const int32_t* __restrict__ neid,
                                               const float* __restrict__ q_t, int k, const int32_t* __restrict__ cnt,
                                               const int32_t* __restrict__ pair_off, const T* __restrict__ mem,
                                               const float* __restrict__ x, const float* __restrict__ tw,
                                               const float* __restrict__ tb, int dm, int de, int dt, int bf16,
                                               float* __restrict__ kv_in, int32_t* __restrict__ pair_nbr,
                                               float* __restrict__ pair_delta) {
  const int Dkv = dm + de + dt;
  const int c = cnt[q];
  const int64_t off = pair_off[q];
  const float tau = q_t[q];
  // lane j < c holds slot j's node, edge and time difference
  const int32_t my_nb = lane < c ? nbr[q * k + lane] : 0;
  const int32_t my_e = lane < c ? neid[q * k + lane] : 0;
  const float my_delta = lane < c ? tau - nt[q * k + lane] : 0.f;
  if (lane < c) {
    pair_nbr[off + lane] = my_nb;
    pair_delta[off + lane] = my_delta;
  }
  for (int j0 = 0; j0 < c; j0 += GATHER_CHUNK) {
    int64_t nb[GATHER_CHUNK];
#pragma unroll
    for (int u = 0; u < GATHER_CHUNK; ++u) nb[u] = __shfl(my_nb, j0 + u, 64);
    for (int c0 = 0; c0 < dm; c0 += 64) {
      const int cc = c0 + lane;
      float v[GATHER_CHUNK];
#pragma unroll
      for (int u = 0; u < GATHER_CHUNK; ++u) v[u] = (j0 + u < c && cc < dm) ? Elem<T>::load(mem, nb[u] * dm + cc) : 0.f;
#pragma unroll
      for (int u = 0; u < GATHER_CHUNK; ++u)
        if (j0 + u < c && cc < dm) kv_in[(off + j0 + u) * Dkv + cc] = v[u];
    }
    if (de > 0) {
      for (int c0 = 0; c0 < de; c0 += 64) {
        const int cc = c0 + lane;
        float v[GATHER_CHUNK];
#pragma unroll
        for (int u = 0; u < GATHER_CHUNK; ++u) {
          const int64_t e = __shfl(my_e, j0 + u, 64);
          v[u] = (j0 + u < c && cc < de) ? x[e * de + cc] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < GATHER_CHUNK; ++u)
          if (j0 + u < c && cc < de) kv_in[(off + j0 + u) * Dkv + dm + cc] = pack_val(v[u], bf16);
      }
    }
    for (int u = 0; u < GATHER_CHUNK; ++u) {
      if (j0 + u >= c) break;
      const float delta = __shfl(my_delta, j0 + u, 64);
      const int64_t row = off + j0 + u;
      for (int jj = lane; jj < dt; jj += 64) {
        const float arg = time_arg(tw[jj], delta, tb[jj]);
        kv_in[row * Dkv + dm + de + jj] = bf16 ? round_to_bf16(cos_for_bf16(arg)) : cosf(arg);
      }
    }
  }
}

// Wave per query: its query-side input and its valid slots' rows, in one launch.
struct GatherArgs {
  const int32_t *q_node, *nbr, *neid, *n_q, *cnt, *pair_off;
  const float *nt, *q_t, *x, *tw, *tb;
  int64_t max_q;
  int k, dm, de, dt, da, bf16;
  float *q_in, *m_in, *kv_in, *pair_delta;
  int32_t* pair_nbr;
};

template <typename T>
__global__ __launch_bounds__(256) void k_attn_gather(GatherArgs a, const T* __restrict__ mem) {
  const int64_t q = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (q >= eff_count(a.max_q, a.n_q)) return;
  gather_q_body<T>(q, lane, a.q_node, mem, a.tw, a.tb, a.dm, a.dt, a.da, a.bf16, a.q_in, a.m_in);
  gather_kv_body<T>(q, lane, a.nbr, a.nt, a.neid, a.q_t, a.k, a.cnt, a.pair_off, mem, a.x, a.tw, a.tb, a.dm, a.de,
                    a.dt, a.bf16, a.kv_in, a.pair_nbr, a.pair_delta);
}

// Float32 fast path (widths divisible by 4): the values of k_attn_gather<float>, computed the same
// way, with a query's rows cut into 4-float groups laid out flat across the wave, so that each lane
// moves 16 bytes per load or store: the query row in one pass, then the memory groups of all its
// valid slots (loads issued GV_UNROLL passes at a time before any store), their edge-feature groups
// the same way, then the time-encoding groups (four cosines per lane).  The time encoder's weights
// and phases are staged in LDS once per block: read from global memory next to each cosine, every
// group waited for its own loads (the cosine's branches keep the next loads from being hoisted).
constexpr int GV_UNROLL = 4;
constexpr int GV_MAX_DT = 256;   // time-encoder width of the fast path (its LDS stage)

// Four consecutive values of a memory row (float32, or bfloat16 widened exactly).
__device__ __forceinline__ float4 load4(const float* p) { return *(const float4*)p; }
__device__ __forceinline__ float4 load4(const uint16_t* p) {
  const uint2 u = *(const uint2*)p;
  return make_float4(bf16_to_f32((uint16_t)(u.x & 0xffffu)), bf16_to_f32((uint16_t)(u.x >> 16)),
                     bf16_to_f32((uint16_t)(u.y & 0xffffu)), bf16_to_f32((uint16_t)(u.y >> 16)));
}
// A time-encoding value as it enters the product (bfloat16 mode: rounded, decided on the correctly
// rounded cosine).
__device__ __forceinline__ float enc_val(float arg, int bf16) {
  return bf16 ? round_to_bf16(cos_for_bf16(arg)) : cosf(arg);
}
__device__ __forceinline__ float4 pack4(float4 v, int bf16) {
  return bf16 ? make_float4(round_to_bf16(v.x), round_to_bf16(v.y), round_to_bf16(v.z), round_to_bf16(v.w)) : v;
}

template <typename T>
__global__ __launch_bounds__(256) void k_attn_gather_v4(GatherArgs a, const T* __restrict__ mem) {
  __shared__ float enc_wb[2 * GV_MAX_DT];   // the time encoder's w, then b
  const int64_t q = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int dm = a.dm, dt = a.dt, da = a.da, de = a.de, gm = dm >> 2, gt = dt >> 2, ge = de >> 2;
  if (dt > 0) {   // every thread stores (slots past 2 dt hold copies that are never read)
    for (int i0 = 0; i0 < 2 * dt; i0 += 256) {
      const int i = i0 + (int)threadIdx.x;
      const int iw = i < dt ? i : dt - 1, ib = i < dt ? 0 : (i - dt < dt ? i - dt : dt - 1);
      const float w = a.tw[iw], b = a.tb[ib];
      enc_wb[i < 2 * GV_MAX_DT ? i : 2 * GV_MAX_DT - 1] = i < dt ? w : b;
    }
  }
  __syncthreads();
  if (q >= eff_count(a.max_q, a.n_q)) return;
  const float* tw = enc_wb;
  const float* tb = enc_wb + dt;
  const int Dq = dm + dt, D = dm + de + dt;   // row widths of q_in and kv_in
  // every per-query scalar first, so that their loads overlap the query row's
  const int64_t node = a.q_node[q];
  const int c = a.cnt[q];
  const int64_t off = a.pair_off[q];
  const float tau = a.q_t[q];
  // loaded on lane < k (in bounds of the [max_q, k] arrays), so they need not wait for c
  const int32_t nb_raw = lane < a.k ? a.nbr[q * a.k + lane] : 0;
  const float t_raw = lane < a.k ? a.nt[q * a.k + lane] : 0.f;
  const int32_t e_raw = lane < a.k && de > 0 ? a.neid[q * a.k + lane] : 0;
  const int32_t my_nb = lane < c ? nb_raw : 0;
  const int32_t my_e = lane < c ? e_raw : 0;
  const float my_t = lane < c ? t_raw : 0.f;
  {
    for (int g = lane; g < gm + gt; g += 64) {
      if (g < gm) {
        const float4 v = load4(mem + node * dm + 4 * g);
        *(float4*)(a.q_in + q * Dq + 4 * g) = v;
        *(float4*)(a.m_in + q * (da + dm) + da + 4 * g) = v;
      } else {
        const int j = 4 * (g - gm);
        float4 o;
        o.x = enc_val(time_arg(tw[j], 0.f, tb[j]), a.bf16);
        o.y = enc_val(time_arg(tw[j + 1], 0.f, tb[j + 1]), a.bf16);
        o.z = enc_val(time_arg(tw[j + 2], 0.f, tb[j + 2]), a.bf16);
        o.w = enc_val(time_arg(tw[j + 3], 0.f, tb[j + 3]), a.bf16);
        *(float4*)(a.q_in + q * Dq + dm + j) = o;
      }
    }
  }
  const float my_delta = lane < c ? tau - my_t : 0.f;
  if (lane < c) {
    a.pair_nbr[off + lane] = my_nb;
    a.pair_delta[off + lane] = my_delta;
  }
  const int nm = c * gm;
  for (int e0 = 0; e0 < nm; e0 += 64 * GV_UNROLL) {
    float4 v[GV_UNROLL];
    int64_t dst[GV_UNROLL];
#pragma unroll
    for (int u = 0; u < GV_UNROLL; ++u) {
      const int e = e0 + 64 * u + lane;
      const int ec = e < nm ? e : nm - 1;   // a valid group, stored only when e < nm
      const int sl = ec / gm, g = ec - sl * gm;
      const int64_t nb = __shfl(my_nb, sl, 64);
      v[u] = load4(mem + nb * dm + 4 * g);
      dst[u] = (off + sl) * D + 4 * g;
    }
#pragma unroll
    for (int u = 0; u < GV_UNROLL; ++u)
      if (e0 + 64 * u + lane < nm) *(float4*)(a.kv_in + dst[u]) = v[u];
  }
  const int nx = c * ge;
  for (int e0 = 0; e0 < nx; e0 += 64 * GV_UNROLL) {   // edge features [dm, dm + de)
    float4 v[GV_UNROLL];
    int64_t dst[GV_UNROLL];
#pragma unroll
    for (int u = 0; u < GV_UNROLL; ++u) {
      const int e = e0 + 64 * u + lane;
      const int ec = e < nx ? e : nx - 1;
      const int sl = ec / ge, g = ec - sl * ge;
      const int64_t eid = __shfl(my_e, sl, 64);
      v[u] = pack4(*(const float4*)(a.x + eid * de + 4 * g), a.bf16);
      dst[u] = (off + sl) * D + dm + 4 * g;
    }
#pragma unroll
    for (int u = 0; u < GV_UNROLL; ++u)
      if (e0 + 64 * u + lane < nx) *(float4*)(a.kv_in + dst[u]) = v[u];
  }
  const int ntg = c * gt;
  for (int e0 = 0; e0 < ntg; e0 += 64) {
    const int e = e0 + lane;
    const int ec = e < ntg ? e : ntg - 1;
    const int sl = ec / gt, g = ec - sl * gt;
    const float delta = __shfl(my_delta, sl, 64);
    if (e < ntg) {
      const int j = 4 * g;
      float4 o;
      o.x = enc_val(time_arg(tw[j], delta, tb[j]), a.bf16);
      o.y = enc_val(time_arg(tw[j + 1], delta, tb[j + 1]), a.bf16);
      o.z = enc_val(time_arg(tw[j + 2], delta, tb[j + 2]), a.bf16);
      o.w = enc_val(time_arg(tw[j + 3], delta, tb[j + 3]), a.bf16);
      *(float4*)(a.kv_in + (off + sl) * D + dm + de + j) = o;
    }
  }
}

constexpr int MAX_DH_CHUNKS = 2;   // head width <= 128

constexpr int SLOT_CHUNK = 8;   // slots whose rows are loaded together (their loads in flight at once)

// Wave per query: softmax over the valid slots of each head, then the
// probability-weighted sum of the values.  Lane j < cnt holds slot j's score.
// Slot rows are read SLOT_CHUNK at a time, all loads issued before use; the
// per-slot sums keep their order.  (The backward below groups the value-row
// loads of its first phase only: grouping the second phase measured slower.)
template <int DHC>   // 64-wide chunks of a head (DHC 64 >= dh)
__global__ __launch_bounds__(256) void k_attn_core(const float* __restrict__ qv, const float* __restrict__ KV,
                                                   const int32_t* __restrict__ cnt,
                                                   const int32_t* __restrict__ pair_off,
                                                   const int32_t* __restrict__ n_q, int64_t max_q, int k, int da,
                                                   int H, int bf16, float* __restrict__ P, float* __restrict__ attn) {
  const int64_t q = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (q >= eff_count(max_q, n_q)) return;
  const int dh = da / H;
  const float scale = 1.0f / sqrtf((float)dh);
  const int c = cnt[q];
  const int64_t off = pair_off[q];
  for (int h = 0; h < H; ++h) {
    float qd[DHC];
#pragma unroll
    for (int cc = 0; cc < DHC; ++cc) {
      const int d = lane + 64 * cc;
      qd[cc] = d < dh ? qv[q * da + h * dh + d] : 0.f;
    }
    float my_s = -INFINITY;
    for (int j0 = 0; j0 < c; j0 += SLOT_CHUNK) {
      float kv[SLOT_CHUNK][DHC];
#pragma unroll
      for (int u = 0; u < SLOT_CHUNK; ++u) {
        const float* Kr = KV + (off + j0 + u) * 2 * da + h * dh;
#pragma unroll
        for (int cc = 0; cc < DHC; ++cc) {
          const int d = lane + 64 * cc;
          kv[u][cc] = (j0 + u < c && d < dh) ? Kr[d] : 0.f;
        }
      }
#pragma unroll
      for (int u = 0; u < SLOT_CHUNK; ++u) {
        if (j0 + u >= c) break;
        float part = 0.f;
#pragma unroll
        for (int cc = 0; cc < DHC; ++cc) part += qd[cc] * kv[u][cc];
        const float sc = wave_sum(part) * scale;
        if (lane == j0 + u) my_s = sc;
      }
    }
    const float m = wave_max(my_s);
    const float e = lane < c ? expf(my_s - m) : 0.f;
    const float den = wave_sum(e);
    const float pj = den > 0.f ? e / den : 0.f;
    if (lane < k) P[(q * H + h) * k + lane] = pj;
    float acc[DHC] = {};
    for (int j0 = 0; j0 < c; j0 += SLOT_CHUNK) {
      float vv[SLOT_CHUNK][DHC];
#pragma unroll
      for (int u = 0; u < SLOT_CHUNK; ++u) {
        const float* Vr = KV + (off + j0 + u) * 2 * da + da + h * dh;
#pragma unroll
        for (int cc = 0; cc < DHC; ++cc) {
          const int d = lane + 64 * cc;
          vv[u][cc] = (j0 + u < c && d < dh) ? Vr[d] : 0.f;
        }
      }
#pragma unroll
      for (int u = 0; u < SLOT_CHUNK; ++u) {
        if (j0 + u >= c) break;
        const float pb = __shfl(pj, j0 + u, 64);
#pragma unroll
        for (int cc = 0; cc < DHC; ++cc) acc[cc] += pb * vv[u][cc];
      }
    }
#pragma unroll
    for (int cc = 0; cc < DHC; ++cc) {
      const int d = lane + 64 * cc;
      if (d < dh) attn[q * da + h * dh + d] = pack_val(acc[cc], bf16);
    }
  }
}

// Wave per query, for one or two heads, d_attn <= 128 and divisible by 4, and at most 2 NP slots.
// A query's K|V rows are contiguous, so each pass takes two slots (slot 2 p + half), 32 lanes per
// slot: lane g of a half holds the row's 4-float group g of K and of V (16-byte loads, all issued
// first; a slot past the count reads row 0, and its products are dropped).  A head's score is the half's 32-lane
// sum of the groups' partial dot products; the softmax runs over each lane's slots and then the two
// halves; the probability-weighted sum of the values stays in the lane of its group, the halves
// added at the end.
template <int NP, int H>
__global__ __launch_bounds__(256) void k_attn_core_v4(const float* __restrict__ qv, const float* __restrict__ KV,
                                                      const int32_t* __restrict__ cnt,
                                                      const int32_t* __restrict__ pair_off,
                                                      const int32_t* __restrict__ n_q, int64_t max_q, int k, int da,
                                                      int bf16, float* __restrict__ P, float* __restrict__ attn) {
  const int64_t q = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (q >= eff_count(max_q, n_q)) return;
  const int half = lane >> 5, g = lane & 31;
  const bool gon = 4 * g < da;
  const int gc = gon ? g : 0;
  const int dh = da / H;
  const float scale = 1.0f / sqrtf((float)dh);
  const int c = cnt[q];
  const int64_t off = pair_off[q];
  const float4 q4 = *(const float4*)(qv + q * da + 4 * gc);
  float4 kr[NP], vr[NP];
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    const int j = 2 * p + half;
    const int64_t row = j < c ? off + j : 0;
    kr[p] = *(const float4*)(KV + row * 2 * da + 4 * gc);
    vr[p] = *(const float4*)(KV + row * 2 * da + da + 4 * gc);
  }
  // head of each element of the group (a group may straddle the head boundary)
  int hd[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) hd[e] = H == 1 ? 0 : (4 * g + e >= dh ? 1 : 0);
  const float qe[4] = {q4.x, q4.y, q4.z, q4.w};
  float pj[NP][H];
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    const float ke[4] = {kr[p].x, kr[p].y, kr[p].z, kr[p].w};
#pragma unroll
    for (int h = 0; h < H; ++h) {
      float v = 0.f;
#pragma unroll
      for (int e = 0; e < 4; ++e) v += (gon && hd[e] == h) ? qe[e] * ke[e] : 0.f;
#pragma unroll
      for (int o = 1; o < 32; o <<= 1) v += __shfl_xor(v, o, 64);
      pj[p][h] = v * scale;
    }
  }
#pragma unroll
  for (int h = 0; h < H; ++h) {
    float m = -INFINITY;
#pragma unroll
    for (int p = 0; p < NP; ++p)
      if (2 * p + half < c) m = fmaxf(m, pj[p][h]);
    m = fmaxf(m, __shfl_xor(m, 32, 64));
    float den = 0.f;
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      pj[p][h] = 2 * p + half < c ? expf(pj[p][h] - m) : 0.f;
      den += pj[p][h];
    }
    den += __shfl_xor(den, 32, 64);
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      pj[p][h] = den > 0.f ? pj[p][h] / den : 0.f;
      const int j = 2 * p + half;
      if (g == 0 && j < k) P[(q * H + h) * k + j] = pj[p][h];
    }
  }
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    const float ve[4] = {vr[p].x, vr[p].y, vr[p].z, vr[p].w};
    const bool on = 2 * p + half < c;   // a slot past the count read row 0, whatever it holds
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float t = ((H == 1 || hd[e] == 0) ? pj[p][0] : pj[p][H - 1]) * ve[e];
      acc[e] += on ? t : 0.f;
    }
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) acc[e] += __shfl_xor(acc[e], 32, 64);
  if (half == 0 && gon) {
    float4 o;
    o.x = pack_val(acc[0], bf16);
    o.y = pack_val(acc[1], bf16);
    o.z = pack_val(acc[2], bf16);
    o.w = pack_val(acc[3], bf16);
    *(float4*)(attn + q * da + 4 * g) = o;
  }
}

// Wave per query: gradients of the softmax-weighted sum and of the scores.
//   dV_j = p_j da_h;  dp_j = da_h . V_j;  ds_j = p_j (dp_j - sum_i p_i dp_i)
//   dq_h = sum_j ds_j K_jh / sqrt(dh);  dK_j = ds_j q_h / sqrt(dh)
template <int DHC>   // 64-wide chunks of a head (DHC 64 >= dh)
__global__ __launch_bounds__(256) void k_attn_core_bwd(const float* __restrict__ qv, const float* __restrict__ KV,
                                                       const float* __restrict__ P, const float* __restrict__ dattn,
                                                       const int32_t* __restrict__ cnt,
                                                       const int32_t* __restrict__ pair_off,
                                                       const int32_t* __restrict__ n_q, int64_t max_q, int k, int da,
                                                       int H, float* __restrict__ dKV, float* __restrict__ dqv) {
  const int64_t q = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (q >= eff_count(max_q, n_q)) return;
  const int dh = da / H;
  const float scale = 1.0f / sqrtf((float)dh);
  const int c = cnt[q];
  const int64_t off = pair_off[q];
  for (int h = 0; h < H; ++h) {
    float qd[DHC], gd[DHC];
#pragma unroll
    for (int cc = 0; cc < DHC; ++cc) {
      const int d = lane + 64 * cc;
      qd[cc] = d < dh ? qv[q * da + h * dh + d] : 0.f;
      gd[cc] = d < dh ? dattn[q * da + h * dh + d] : 0.f;
    }
    const float pl = lane < c ? P[(q * H + h) * k + lane] : 0.f;
    float my_dp = 0.f;
    for (int j0 = 0; j0 < c; j0 += SLOT_CHUNK) {   // value rows of SLOT_CHUNK slots loaded together
      float vv[SLOT_CHUNK][DHC];
#pragma unroll
      for (int u = 0; u < SLOT_CHUNK; ++u) {
        const float* Vr = KV + (off + j0 + u) * 2 * da + da + h * dh;
#pragma unroll
        for (int cc = 0; cc < DHC; ++cc) {
          const int d = lane + 64 * cc;
          vv[u][cc] = (j0 + u < c && d < dh) ? Vr[d] : 0.f;
        }
      }
#pragma unroll
      for (int u = 0; u < SLOT_CHUNK; ++u) {
        if (j0 + u >= c) break;
        float part = 0.f;
#pragma unroll
        for (int cc = 0; cc < DHC; ++cc) part += gd[cc] * vv[u][cc];
        const float dp = wave_sum(part);
        if (lane == j0 + u) my_dp = dp;
      }
    }
    const float sdp = wave_sum(pl * my_dp);
    const float dsl = pl * (my_dp - sdp);
    float dq[DHC] = {};
    for (int j = 0; j < c; ++j) {
      const float dsj = __shfl(dsl, j, 64);
      const float pj = __shfl(pl, j, 64);
      const int64_t row = off + j;
      const float* Kr = KV + row * 2 * da + h * dh;
      float* dK = dKV + row * 2 * da + h * dh;
#pragma unroll
      for (int cc = 0; cc < DHC; ++cc) {
        const int d = lane + 64 * cc;
        if (d < dh) {
          dq[cc] += dsj * Kr[d];
          dK[d] = dsj * qd[cc] * scale;
          dK[da + d] = pj * gd[cc];
        }
      }
    }
#pragma unroll
    for (int cc = 0; cc < DHC; ++cc) {
      const int d = lane + 64 * cc;
      if (d < dh) dqv[q * da + h * dh + d] = dq[cc] * scale;
    }
  }
}

// The backward of k_attn_core_v4 in its layout (two slots per pass, lane g of a half holding
// 4-float group g of K, V, q and dattn): dp per slot and head as a 32-lane sum, the softmax
// backward over each lane's slots and the two halves, dK and dV of a slot stored by the lanes of
// its half as 16-byte groups, dq summed over each lane's slots and then the halves.  A slot past
// the count reads row 0, and every value it could contribute is dropped by a select.
template <int NP, int H>
__global__ __launch_bounds__(256) void k_attn_core_bwd_v4(const float* __restrict__ qv, const float* __restrict__ KV,
                                                          const float* __restrict__ P,
                                                          const float* __restrict__ dattn,
                                                          const int32_t* __restrict__ cnt,
                                                          const int32_t* __restrict__ pair_off,
                                                          const int32_t* __restrict__ n_q, int64_t max_q, int k,
                                                          int da, float* __restrict__ dKV, float* __restrict__ dqv) {
  const int64_t q = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (q >= eff_count(max_q, n_q)) return;
  const int half = lane >> 5, g = lane & 31;
  const bool gon = 4 * g < da;
  const int gc = gon ? g : 0;
  const int dh = da / H;
  const float scale = 1.0f / sqrtf((float)dh);
  const int c = cnt[q];
  const int64_t off = pair_off[q];
  const float4 q4 = *(const float4*)(qv + q * da + 4 * gc);
  const float4 g4 = *(const float4*)(dattn + q * da + 4 * gc);
  float4 kr[NP], vr[NP];
  float pp[NP][H];
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    const int j = 2 * p + half;
    const bool on = j < c;
    const int64_t row = on ? off + j : 0;
    kr[p] = *(const float4*)(KV + row * 2 * da + 4 * gc);
    vr[p] = *(const float4*)(KV + row * 2 * da + da + 4 * gc);
#pragma unroll
    for (int h = 0; h < H; ++h) {
      const float v = P[(q * H + h) * k + (on ? j : 0)];
      pp[p][h] = on ? v : 0.f;
    }
  }
  int hd[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) hd[e] = H == 1 ? 0 : (4 * g + e >= dh ? 1 : 0);
  const float qe[4] = {q4.x, q4.y, q4.z, q4.w};
  const float ge[4] = {g4.x, g4.y, g4.z, g4.w};
  // dp_j = dattn_h . V_j (32-lane sums), then sdp_h = sum_j p_j dp_j over both halves
  float ds[NP][H];
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    const float ve[4] = {vr[p].x, vr[p].y, vr[p].z, vr[p].w};
    const bool on = 2 * p + half < c;
#pragma unroll
    for (int h = 0; h < H; ++h) {
      float v = 0.f;
#pragma unroll
      for (int e = 0; e < 4; ++e) v += (gon && hd[e] == h) ? ge[e] * ve[e] : 0.f;
#pragma unroll
      for (int o = 1; o < 32; o <<= 1) v += __shfl_xor(v, o, 64);
      ds[p][h] = on ? v : 0.f;
    }
  }
#pragma unroll
  for (int h = 0; h < H; ++h) {
    float sdp = 0.f;
#pragma unroll
    for (int p = 0; p < NP; ++p) sdp += pp[p][h] * ds[p][h];
    sdp += __shfl_xor(sdp, 32, 64);
#pragma unroll
    for (int p = 0; p < NP; ++p) ds[p][h] = pp[p][h] * (ds[p][h] - sdp);
  }
  float dq[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    const int j = 2 * p + half;
    const bool on = j < c;
    const float ke[4] = {kr[p].x, kr[p].y, kr[p].z, kr[p].w};
    float dk[4], dv[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float dsh = (H == 1 || hd[e] == 0) ? ds[p][0] : ds[p][H - 1];
      const float ph = (H == 1 || hd[e] == 0) ? pp[p][0] : pp[p][H - 1];
      const float t = dsh * ke[e];
      dq[e] += on ? t : 0.f;
      dk[e] = dsh * qe[e] * scale;
      dv[e] = ph * ge[e];
    }
    if (on && gon) {
      float* dst = dKV + (off + j) * 2 * da + 4 * g;
      *(float4*)dst = make_float4(dk[0], dk[1], dk[2], dk[3]);
      *(float4*)(dst + da) = make_float4(dv[0], dv[1], dv[2], dv[3]);
    }
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) dq[e] += __shfl_xor(dq[e], 32, 64);
  if (half == 0 && gon)
    *(float4*)(dqv + q * da + 4 * g) =
        make_float4(dq[0] * scale, dq[1] * scale, dq[2] * scale, dq[3] * scale);
}

// [dW_k; dW_v] and [db_k; db_v] from the stacked weight gradient.
__global__ void k_split_kv_grads(const float* __restrict__ dW, const float* __restrict__ db, int da, int Dkv,
                                 float* __restrict__ dWk, float* __restrict__ dWv, float* __restrict__ dbk,
                                 float* __restrict__ dbv) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t half = (int64_t)da * Dkv;
  if (e < half) {
    dWk[e] = dW[e];
    dWv[e] = dW[half + e];
  }
  if (e < da) {
    dbk[e] = db[e];
    dbv[e] = db[da + e];
  }
}

// ---------------------------------------------------------------- d M' by node (deterministic)

// Node -> row map for the rows updated this step, plus empty segment bounds.
// The map lives in the workspace and is not cleared: a lookup is accepted only
// if it names a row r < n_rows with uniq[r] equal to the node, so stale
// entries are rejected.
__global__ void k_row_map(const int32_t* __restrict__ uniq, const int32_t* __restrict__ n_rows, int64_t max_rows,
                          int32_t* __restrict__ row_of, int32_t* __restrict__ seg_lo, int32_t* __restrict__ seg_hi) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= max_rows) return;
  seg_lo[r] = 0;   // empty segments until k_seg_bounds records the real ones
  seg_hi[r] = 0;
  if (r < eff_count(max_rows, n_rows)) row_of[uniq[r]] = (int32_t)r;
}

// Occurrence o < max_q is query o; o = max_q + p is compact slot p.  Its key is
// the row of its node among the rows updated this step, or `sentinel` when
// the node was not updated, or the query / slot is beyond the device counts.
// Threads o >= max_q walk the sampled grid (query q, slot j): the valid slots of a query are the
// prefix of its list, so slot j < cnt[q] is compact slot pair_off[q] + j, and the thread for grid
// index i also fills compact position i when i is past the valid count.  Every position is written
// once, from the sampler's output and the slot counts alone (no forward gather needed).
__device__ __forceinline__ uint32_t occ_key(int64_t node, const int32_t* __restrict__ uniq, int32_t rows,
                                            const int32_t* __restrict__ row_of, uint32_t sentinel) {
  if (node < 0) return sentinel;
  const int32_t r = row_of[node];
  return (r >= 0 && r < rows && uniq[r] == node) ? (uint32_t)r : sentinel;
}

__global__ void k_occ_keys(const int32_t* __restrict__ q_node, const int32_t* __restrict__ nbr,
                           const int32_t* __restrict__ cnt, const int32_t* __restrict__ pair_off,
                           const int32_t* __restrict__ n_q, int64_t max_q, int k,
                           const int32_t* __restrict__ n_valid, int64_t max_p, const int32_t* __restrict__ uniq,
                           const int32_t* __restrict__ n_rows, int64_t max_rows, const int32_t* __restrict__ row_of,
                           uint32_t sentinel, uint32_t* __restrict__ keys, uint32_t* __restrict__ vals) {
  const int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (o >= max_q + max_p) return;
  const int32_t rows = (int32_t)eff_count(max_rows, n_rows);
  if (o < max_q) {
    keys[o] = occ_key(o < eff_count(max_q, n_q) ? q_node[o] : -1, uniq, rows, row_of, sentinel);
    vals[o] = (uint32_t)o;
    return;
  }
  const int64_t i = o - max_q;
  const int64_t q = i / k;
  const int j = (int)(i - q * k);
  if (j < cnt[q]) {
    const int64_t p = max_q + pair_off[q] + j;
    keys[p] = occ_key(nbr[i], uniq, rows, row_of, sentinel);
    vals[p] = (uint32_t)p;
  }
  if (i >= eff_count(max_p, n_valid)) {
    keys[o] = sentinel;
    vals[o] = (uint32_t)o;
  }
}

// seg_lo[row], seg_hi[row]: the sorted positions [lo, hi) holding row's occurrences.
__global__ void k_seg_bounds(const uint32_t* __restrict__ keys, int64_t n, uint32_t sentinel,
                             int32_t* __restrict__ seg_lo, int32_t* __restrict__ seg_hi) {
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= n) return;
  const uint32_t k = keys[p];
  if (k == sentinel) return;
  if (p == 0 || keys[p - 1] != k) seg_lo[k] = (int32_t)p;
  if (p == n - 1 || keys[p + 1] != k) seg_hi[k] = (int32_t)(p + 1);
}

constexpr int SEG_TILE = 64;     // sorted occurrences per wave (the attention's d M')
constexpr int SEG_TILE_ROWS = 16;   // the same for segsum_rows (few occurrences: more, shorter waves)

struct SegCtx {
  const uint32_t* keys;
  const uint32_t* vals;
  int64_t n_occ;
  uint32_t sentinel;
  int64_t max_q;
  const float* dhq;   // [Q, ldq] query-side gradient of M[q] (columns [0, dm))
  int64_t ldq;
  const float* dkv;   // [P, 2 da] compact-slot gradient of (K, V)
  int dm, w2;         // w2 = 2 da ; row width W = dm + w2
  float* S;           // [rows, W] complete sums (columns [0, dm) go to D instead)
  float* D;           // [rows, dm] d M' itself: the dh_q sums land there, the dK|dV product adds to them
  float* head;        // [ntiles, W]
  float* tail;        // [ntiles, W]
  const int32_t* seg_lo;   // [rows] first sorted position of the row
  const int32_t* seg_hi;   // [rows] one past its last
  int tile;                // sorted positions per wave (at most 64)
};

// A complete row of sums: columns < dm to D, the rest to S.
template <int NC>
__device__ __forceinline__ void seg_store_row(const SegCtx& c, int64_t row, const float* acc, int lane) {
  const int W = c.dm + c.w2;
#pragma unroll
  for (int i = 0; i < NC; ++i) {
    const int col = lane + 64 * i;
    if (col < c.dm) c.D[row * c.dm + col] = acc[i];
    else if (col < W) c.S[row * W + col] = acc[i];
  }
}

// The row of occurrence o over the lanes, NC column chunks (zero outside its columns).
template <int NC>
__device__ __forceinline__ void seg_row_nc(const SegCtx& c, uint32_t o, float* r, int lane) {
  const int W = c.dm + c.w2;
  if ((int64_t)o < c.max_q) {
    const float* src = c.dhq + (int64_t)o * c.ldq;
#pragma unroll
    for (int i = 0; i < NC; ++i) {
      const int col = lane + 64 * i;
      r[i] = col < c.dm ? src[col] : 0.f;
    }
  } else {
    const float* src = c.dkv + ((int64_t)o - c.max_q) * c.w2;
#pragma unroll
    for (int i = 0; i < NC; ++i) {
      const int col = lane + 64 * i;
      r[i] = (col >= c.dm && col < W) ? src[col - c.dm] : 0.f;
    }
  }
}

// Wave per tile of c.tile (at most 64) sorted positions; lane i holds position
// p0 + i.  The wave walks the positions in order with one running sum,
// loading the rows of SEG_PREFETCH positions at a time (whatever segments
// they belong to); when the key changes, the finished segment is stored.  A
// segment entirely inside the tile goes to S; the piece of one that began
// before the tile goes to head[tile]; the piece of one that continues past it
// goes to tail[tile].  The fixup pass adds the pieces in tile order.  Each
// segment's sum runs over its positions in order.
constexpr int SEG_PREFETCH = 8;

template <int NC>
__global__ __launch_bounds__(256) void k_segsum_tiles(SegCtx c) {
  const int64_t tile = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int64_t p0 = tile * c.tile;
  if (p0 >= c.n_occ) return;
  const int cnt = (int)min((int64_t)c.tile, c.n_occ - p0);
  const int W = c.dm + c.w2;
  const uint32_t my_key = lane < cnt ? c.keys[p0 + lane] : c.sentinel;
  const uint32_t my_val = lane < cnt ? c.vals[p0 + lane] : 0u;
  const uint32_t key_before = p0 > 0 ? c.keys[p0 - 1] : c.sentinel;
  const uint32_t key_after = p0 + cnt < c.n_occ ? c.keys[p0 + cnt] : c.sentinel;
  uint32_t cur = __shfl(my_key, 0, 64);
  if (cur == c.sentinel) return;   // sentinels sort last: nothing in this tile
  int start = 0;
  float acc[NC];
#pragma unroll
  for (int i = 0; i < NC; ++i) acc[i] = 0.f;
  auto flush = [&](int end) {
    const bool before = start == 0 && key_before == cur;
    const bool after = end == cnt && key_after == cur;
    if (!before && !after) {   // the whole segment is in this tile
      seg_store_row<NC>(c, (int64_t)cur, acc, lane);
      return;
    }
    float* dst = before ? c.head + tile * W : c.tail + tile * W;
#pragma unroll
    for (int i = 0; i < NC; ++i) {
      const int col = lane + 64 * i;
      if (col < W) dst[col] = acc[i];
    }
  };
  for (int q0 = 0; q0 < cnt; q0 += SEG_PREFETCH) {
    float r[SEG_PREFETCH][NC];
#pragma unroll
    for (int u = 0; u < SEG_PREFETCH; ++u) {
      const int p = q0 + u;
      const uint32_t k = __shfl(my_key, p, 64);
      const uint32_t o = __shfl(my_val, p, 64);
      if (p < cnt && k != c.sentinel) {
        seg_row_nc<NC>(c, o, r[u], lane);
      } else {
#pragma unroll
        for (int i = 0; i < NC; ++i) r[u][i] = 0.f;
      }
    }
#pragma unroll
    for (int u = 0; u < SEG_PREFETCH; ++u) {
      const int p = q0 + u;
      if (p >= cnt) break;
      const uint32_t k = __shfl(my_key, p, 64);
      if (k != cur) {
        flush(p);
        if (k == c.sentinel) return;
        cur = k;
        start = p;
#pragma unroll
        for (int i = 0; i < NC; ++i) acc[i] = 0.f;
      }
#pragma unroll
      for (int i = 0; i < NC; ++i) acc[i] += r[u][i];
    }
  }
  flush(cnt);
}

// A finished segment's sums (groups qa and qb of this lane): a whole segment to D / S, a piece that
// began before the tile to head[tile], one that continues past it to tail[tile].
__device__ __forceinline__ void seg_flush_v4(const SegCtx& c, int64_t tile, uint32_t cur, bool before, bool after,
                                             int qa, int qb, f32x4 acc_a, f32x4 acc_b) {
  const int W = c.dm + c.w2, W4 = W >> 2, dm4 = c.dm >> 2;
  if (!before && !after) {
    float* row_d = c.D + (int64_t)cur * c.dm;
    float* row_s = c.S + (int64_t)cur * W;
    if (qa < dm4) *(f32x4*)(row_d + 4 * qa) = acc_a;
    else if (qa < W4) *(f32x4*)(row_s + 4 * qa) = acc_a;
    if (qb < dm4) *(f32x4*)(row_d + 4 * qb) = acc_b;
    else if (qb < W4) *(f32x4*)(row_s + 4 * qb) = acc_b;
    return;
  }
  float* dst = before ? c.head + tile * W : c.tail + tile * W;
  if (qa < W4) *(f32x4*)(dst + 4 * qa) = acc_a;
  if (qb < W4) *(f32x4*)(dst + 4 * qb) = acc_b;
}

// A loaded 16-byte group kept in its registers (see keep_live).
__device__ __forceinline__ void keep_live4(f32x4& v) { asm volatile("" : "+v"(v)); }

// k_segsum_tiles with 16-byte groups (d_mem and d_attn divisible by 4, W <= 512): lane l holds
// the row's 4-column groups l and l + 64.  Every column's sum runs over the positions in the same
// order as k_segsum_tiles, so the results are bitwise the same.  The tile's positions are read with
// wave-uniform lane indices, so the keys and row choices are scalar; each prefetched position loads
// one clamped 16-byte group per lane group, unconditionally (a position past the tile's end or past
// its last key re-reads position 0's row), and the groups outside the row are zeroed afterwards.
// With no load under a per-lane test, all of a batch's loads are in flight together.
__global__ __launch_bounds__(256) void k_segsum_tiles_v4(SegCtx c) {
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t tile = (int64_t)blockIdx.x * 4 + wid;
  const int lane = threadIdx.x & 63;
  const int64_t p0 = tile * c.tile;
  if (p0 >= c.n_occ) return;
  const int cnt = (int)min((int64_t)c.tile, c.n_occ - p0);
  const int W = c.dm + c.w2, W4 = W >> 2, dm4 = c.dm >> 2;
  const int qa = lane, qb = lane + 64;   // this lane's column groups
  const uint32_t my_key = lane < cnt ? c.keys[p0 + lane] : c.sentinel;
  const uint32_t my_val = lane < cnt ? c.vals[p0 + lane] : 0u;
  const uint32_t key_before = p0 > 0 ? c.keys[p0 - 1] : c.sentinel;
  const uint32_t key_after = p0 + cnt < c.n_occ ? c.keys[p0 + cnt] : c.sentinel;
  uint32_t cur = (uint32_t)__builtin_amdgcn_readfirstlane((int)my_key);
  if (cur == c.sentinel) return;   // sentinels sort last: nothing in this tile
  const f32x4 z4 = {0.f, 0.f, 0.f, 0.f};
  int start = 0;
  f32x4 acc_a = z4, acc_b = z4;
  for (int q0 = 0; q0 < cnt; q0 += SEG_PREFETCH) {
    f32x4 ra[SEG_PREFETCH], rb[SEG_PREFETCH];
    bool va[SEG_PREFETCH], vb[SEG_PREFETCH];
#pragma unroll
    for (int u = 0; u < SEG_PREFETCH; ++u) {
      const int p = q0 + u;
      const uint32_t k = (uint32_t)__builtin_amdgcn_readlane((int)my_key, p < cnt ? p : 0);
      const bool live = p < cnt && k != c.sentinel;
      const uint32_t o = (uint32_t)__builtin_amdgcn_readlane((int)my_val, live ? p : 0);
      const bool isq = (int64_t)o < c.max_q;
      const float* src = isq ? c.dhq + (int64_t)o * c.ldq : c.dkv + ((int64_t)o - c.max_q) * c.w2 - c.dm;
      const int lo = isq ? 0 : dm4, hi = isq ? dm4 : W4;   // the row's groups: [lo, hi), never empty
      ra[u] = *(const f32x4*)(src + 4 * min(max(qa, lo), hi - 1));
      rb[u] = *(const f32x4*)(src + 4 * min(max(qb, lo), hi - 1));
      va[u] = live && qa >= lo && qa < hi;
      vb[u] = live && qb >= lo && qb < hi;
    }
#pragma unroll
    for (int u = 0; u < SEG_PREFETCH; ++u) {
      keep_live4(ra[u]);
      keep_live4(rb[u]);
    }
#pragma unroll
    for (int u = 0; u < SEG_PREFETCH; ++u) {
      const int p = q0 + u;
      if (p < cnt) {
        const uint32_t k = (uint32_t)__builtin_amdgcn_readlane((int)my_key, p);
        if (k != cur) {
          seg_flush_v4(c, tile, cur, start == 0 && key_before == cur, false, qa, qb, acc_a, acc_b);
          if (k == c.sentinel) return;
          cur = k;
          start = p;
          acc_a = z4;
          acc_b = z4;
        }
        acc_a += va[u] ? ra[u] : z4;
        acc_b += vb[u] ? rb[u] : z4;
      }
    }
  }
  seg_flush_v4(c, tile, cur, start == 0 && key_before == cur, key_after == cur, qa, qb, acc_a, acc_b);
}

// The rows no tile could finish.  Every wave first zeroes, grid-stride, the rows with no occurrence.
// Then block b checks tiles tpb b .. tpb b + tpb - 1 (one lane each, tpb <= 64, about 1024 blocks over
// all tiles, so that a skewed stream's many hub rows spread over many blocks): a tile whose last row starts in it and
// continues past it (rows inside one tile were written whole) has that row summed:
// tail[tile] + head[tile + 1] + ... + head[t1].  A row of more than FIX_WAVES heads is summed by the
// whole block: the waves take interleaved heads, four at a time with all their loads in flight (no
// per-lane test: a chunk past the row's W columns re-reads column W - 1 and is never stored), and their
// partial sums are added in wave order.  A shorter row is summed by one wave.  NC = ceil(W / 64) <= 5.
constexpr int FIX_WAVES = 16;
constexpr int FIX_BLOCKS = 1024;   // blocks the tile checks aim for

template <int NC>
__global__ __launch_bounds__(64 * FIX_WAVES) void k_segsum_fixup(SegCtx c, const int32_t* __restrict__ n_rows,
                                                                 int64_t max_rows, int64_t ntiles, int tpb) {
  __shared__ float part[FIX_WAVES][NC * 64];
  const int64_t blk = blockIdx.x;
  const int lane = threadIdx.x & 63;
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int W = c.dm + c.w2;
  const int64_t rows = eff_count(max_rows, n_rows);
  for (int64_t zr = blk * FIX_WAVES + wid; zr < rows; zr += (int64_t)gridDim.x * FIX_WAVES) {
    if (c.seg_lo[zr] == c.seg_hi[zr]) {   // no occurrence: zero gradient
      float z[NC];
#pragma unroll
      for (int i = 0; i < NC; ++i) z[i] = 0.f;
      seg_store_row<NC>(c, zr, z, lane);
    }
  }
  // the rest depends on the block only (uniform branches around the barriers)
  const int64_t tile0 = blk * tpb;
  if (tile0 >= ntiles) return;
  // lane l: does tile tile0 + l end inside a row that starts in it and continues past it (todo: for more
  // than FIX_WAVES further tiles, shorter: for fewer)?
  uint64_t todo, shorter;
  {
    const int64_t tile = tile0 + lane < ntiles ? tile0 + lane : ntiles - 1;
    const int64_t p_last = min((tile + 1) * c.tile, c.n_occ) - 1;
    const int64_t p_next = p_last + 1 < c.n_occ ? p_last + 1 : p_last;
    const uint32_t key = c.keys[p_last], next = c.keys[p_next];
    const bool cont = lane < tpb && tile0 + lane < ntiles && p_last + 1 < c.n_occ && key != c.sentinel && next == key;
    const bool starts = cont && c.seg_lo[key] >= tile * c.tile;
    const bool longer = starts && (int64_t)(c.seg_hi[key] - 1) / c.tile - tile > FIX_WAVES;
    todo = __ballot(starts && longer);
    shorter = __ballot(starts && !longer);
  }
  int cc[NC];
#pragma unroll
  for (int i = 0; i < NC; ++i) cc[i] = lane + 64 * i < W ? lane + 64 * i : W - 1;
  // Rows with at most FIX_WAVES heads: one wave each (every FIX_WAVES-th such row to this wave).  On
  // the block path each wave would hold at most one head and the parts be added in wave order, so
  // tail + (((0 + head 1) + head 2) + ...) here is the same sum, bit for bit.
  for (int idx = 0; shorter; ++idx) {
    const int l = __builtin_ctzll(shorter);
    shorter &= shorter - 1;
    if (idx % FIX_WAVES != wid) continue;
    const int64_t tile = tile0 + l;
    const int64_t p_last = min((tile + 1) * c.tile, c.n_occ) - 1;
    const uint32_t key = c.keys[p_last];
    const int64_t t1 = (c.seg_hi[key] - 1) / c.tile;
    const float* tl = c.tail + tile * W;
    float acc[NC], tv[NC];
#pragma unroll
    for (int i = 0; i < NC; ++i) {
      tv[i] = tl[cc[i]];
      acc[i] = 0.f;
    }
    for (int64_t t = tile + 1; t <= t1; t += 4) {   // four heads' loads in flight, added in order
      float v[4][NC];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const float* h = c.head + (t + u <= t1 ? t + u : t1) * W;
#pragma unroll
        for (int i = 0; i < NC; ++i) v[u][i] = h[cc[i]];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int i = 0; i < NC; ++i) keep_live(v[u][i]);
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (t + u <= t1) {
#pragma unroll
          for (int i = 0; i < NC; ++i) acc[i] += v[u][i];
        }
    }
#pragma unroll
    for (int i = 0; i < NC; ++i) acc[i] = tv[i] + acc[i];
    seg_store_row<NC>(c, (int64_t)key, acc, lane);
  }
  while (todo) {
    const int l = __builtin_ctzll(todo);
    todo &= todo - 1;
    const int64_t tile = tile0 + l;
    const int64_t p_last = min((tile + 1) * c.tile, c.n_occ) - 1;
    const uint32_t key = c.keys[p_last];
    const int64_t t1 = (c.seg_hi[key] - 1) / c.tile;
    float acc[NC];
#pragma unroll
    for (int i = 0; i < NC; ++i) acc[i] = 0.f;
    int64_t t = tile + 1 + wid;
    constexpr int64_t S4 = 4 * FIX_WAVES;
    for (; t + 3 * FIX_WAVES <= t1; t += S4) {
      const float* h0 = c.head + t * W;
      const float* h1 = h0 + FIX_WAVES * (int64_t)W;
      const float* h2 = h0 + 2 * FIX_WAVES * (int64_t)W;
      const float* h3 = h0 + 3 * FIX_WAVES * (int64_t)W;
      float v[4][NC];
#pragma unroll
      for (int i = 0; i < NC; ++i) {
        v[0][i] = h0[cc[i]];
        v[1][i] = h1[cc[i]];
        v[2][i] = h2[cc[i]];
        v[3][i] = h3[cc[i]];
      }
#pragma unroll
      for (int i = 0; i < NC; ++i) acc[i] += ((v[0][i] + v[1][i]) + v[2][i]) + v[3][i];
    }
    for (; t <= t1; t += FIX_WAVES) {
      const float* h = c.head + t * W;
      float v[NC];
#pragma unroll
      for (int i = 0; i < NC; ++i) v[i] = h[cc[i]];
#pragma unroll
      for (int i = 0; i < NC; ++i) acc[i] += v[i];
    }
#pragma unroll
    for (int i = 0; i < NC; ++i) part[wid][i * 64 + lane] = acc[i];
    __syncthreads();
    if (wid == 0) {
      const float* tl = c.tail + tile * W;
      float tv[NC];
#pragma unroll
      for (int i = 0; i < NC; ++i) tv[i] = tl[cc[i]];
#pragma unroll
      for (int i = 0; i < NC; ++i) {
        const int o = i * 64 + lane;
        float sum = 0.f;
        for (int w = 0; w < FIX_WAVES; ++w) sum += part[w][o];
        acc[i] = tv[i] + sum;
      }
      seg_store_row<NC>(c, (int64_t)key, acc, lane);
    }
    __syncthreads();   // part is free for the next row
  }
}

// Rows of 321 to 512 columns: the same sums with a per-chunk test around each load (the batched
// form above would need more than the 128 registers a thread of a 1024-thread block has).
constexpr int FIX_WIDE_C = 8;

__global__ __launch_bounds__(64 * FIX_WAVES) void k_segsum_fixup_wide(SegCtx c, const int32_t* __restrict__ n_rows,
                                                                      int64_t max_rows, int64_t ntiles) {
  __shared__ float part[FIX_WAVES][FIX_WIDE_C * 64];
  const int64_t blk = blockIdx.x;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int W = c.dm + c.w2;
  const int64_t zr = blk * FIX_WAVES + wid;
  if (zr < eff_count(max_rows, n_rows) && c.seg_lo[zr] == c.seg_hi[zr]) {   // no occurrence: zero gradient
    float z[FIX_WIDE_C];
#pragma unroll
    for (int i = 0; i < FIX_WIDE_C; ++i) z[i] = 0.f;
    seg_store_row<FIX_WIDE_C>(c, zr, z, lane);
  }
  // the rest depends on the block only (uniform branches around the barrier)
  if (blk >= ntiles) return;
  const int64_t p_last = min((blk + 1) * c.tile, c.n_occ) - 1;
  if (p_last + 1 >= c.n_occ) return;
  const uint32_t key = c.keys[p_last];
  if (key == c.sentinel || c.keys[p_last + 1] != key) return;
  if (c.seg_lo[key] < blk * c.tile) return;   // started in an earlier tile, whose block sums it
  const int64_t t1 = (c.seg_hi[key] - 1) / c.tile;
  float acc[FIX_WIDE_C];
#pragma unroll
  for (int i = 0; i < FIX_WIDE_C; ++i) acc[i] = 0.f;
  int64_t t = blk + 1 + wid;
  constexpr int64_t S4 = 4 * FIX_WAVES;
  for (; t + 3 * FIX_WAVES <= t1; t += S4) {
    const float* h0 = c.head + t * W;
    const float* h1 = h0 + FIX_WAVES * (int64_t)W;
    const float* h2 = h0 + 2 * FIX_WAVES * (int64_t)W;
    const float* h3 = h0 + 3 * FIX_WAVES * (int64_t)W;
#pragma unroll
    for (int i = 0; i < FIX_WIDE_C; ++i) {
      const int col = lane + 64 * i;
      if (col < W) acc[i] += ((h0[col] + h1[col]) + h2[col]) + h3[col];
    }
  }
  for (; t <= t1; t += FIX_WAVES) {
    const float* h = c.head + t * W;
#pragma unroll
    for (int i = 0; i < FIX_WIDE_C; ++i) {
      const int col = lane + 64 * i;
      if (col < W) acc[i] += h[col];
    }
  }
#pragma unroll
  for (int i = 0; i < FIX_WIDE_C; ++i) part[wid][i * 64 + lane] = acc[i];
  __syncthreads();
  if (wid != 0) return;
  const float* tl = c.tail + blk * W;
#pragma unroll
  for (int i = 0; i < FIX_WIDE_C; ++i) {
    const int col = lane + 64 * i;
    const int o = i * 64 + lane;
    if (col < W) {
      float sum = 0.f;
      for (int w = 0; w < FIX_WAVES; ++w) sum += part[w][o];
      acc[i] = tl[col] + sum;
    }
  }
  seg_store_row<FIX_WIDE_C>(c, (int64_t)key, acc, lane);
}

// The fixup over max_rows rows and ntiles tiles (its grid covers both), with ceil(W / 64) column chunks.
void launch_segsum_fixup(const SegCtx& c, const int32_t* n_rows, int64_t max_rows, int64_t ntiles, hipStream_t s) {
  const unsigned b = 64 * FIX_WAVES;
  if (cdiv(c.dm + c.w2, 64) > 5) {   // one block per tile (and per FIX_WAVES rows)
    const int64_t nfix = ntiles > cdiv(max_rows, FIX_WAVES) ? ntiles : cdiv(max_rows, FIX_WAVES);
    k_segsum_fixup_wide<<<(unsigned)nfix, b, 0, s>>>(c, n_rows, max_rows, ntiles);
    return;
  }
  // tpb tiles per block (about FIX_BLOCKS blocks), and at least enough blocks for the row zeroing to take a
  // few rows per wave
  const int64_t tpb64 = cdiv(ntiles, FIX_BLOCKS);
  const int tpb = (int)(tpb64 < 1 ? 1 : (tpb64 > 64 ? 64 : tpb64));
  const int64_t zb = cdiv(max_rows, FIX_WAVES) < FIX_BLOCKS ? cdiv(max_rows, FIX_WAVES) : FIX_BLOCKS;
  const int64_t tb = cdiv(ntiles, tpb);
  const unsigned g = (unsigned)(tb > zb ? tb : (zb > 0 ? zb : 1));
  switch (cdiv(c.dm + c.w2, 64)) {
    case 1: k_segsum_fixup<1><<<g, b, 0, s>>>(c, n_rows, max_rows, ntiles, tpb); break;
    case 2: k_segsum_fixup<2><<<g, b, 0, s>>>(c, n_rows, max_rows, ntiles, tpb); break;
    case 3: k_segsum_fixup<3><<<g, b, 0, s>>>(c, n_rows, max_rows, ntiles, tpb); break;
    case 4: k_segsum_fixup<4><<<g, b, 0, s>>>(c, n_rows, max_rows, ntiles, tpb); break;
    default: k_segsum_fixup<5><<<g, b, 0, s>>>(c, n_rows, max_rows, ntiles, tpb); break;
  }
}

struct BwdWs {
  float *dm1, *dm_in, *dattn, *dqv, *dKV, *tg_part, *tg_part2, *S, *head, *tail, *dWkv, *dbkv;
  char* scratch_merge;    // split-K partials of the output and merge layers' weight gradients (their own:
  size_t scratch_merge_bytes;   // with a second stream they run there, beside the other products)
  uint32_t *keys, *vals;
  int32_t *seg_lo, *seg_hi, *row_of;
  char* scratch;          // split-K partials of the parameter-gradient products
  size_t scratch_bytes;
  char* sort_scratch;     // radix sort of the dM' grouping (disjoint: the two parts may run concurrently)
  size_t sort_scratch_bytes;
  size_t total;
};

// The output and merge layers' weight gradients apart from the query layer's, on the second stream when
// there is one, from this many query rows on (at a few thousand rows that batch, beside the score
// backward and the query projection's data gradient, slowed them more than it saved: 7.98 -> 7.80 M
// events/s on the skewed stream, 12,000 queries; 6.35 -> 6.73 M at 180,000).
constexpr int64_t MERGE_DW_APART_ROWS = 65536;
bool merge_dw_apart(int64_t Q) { return Q >= MERGE_DW_APART_ROWS; }

BwdWs carve_bwd(void* base, const AttnShape& s, int64_t max_rows) {
  char* w = (char*)base;
  BwdWs v;
  auto take = [&](size_t bytes) { char* r = w; w += a256(bytes); return r; };
  const int64_t n_occ = s.Q + s.P;
  const int64_t ntiles = cdiv(n_occ, SEG_TILE);
  const int W = s.dm + 2 * s.da;
  const int64_t dtp = s.dt > 0 ? s.dt : 1;
  v.dm1 = (float*)take(sizeof(float) * s.Q * s.da);
  v.dm_in = (float*)take(sizeof(float) * s.Q * (s.da + s.dm));
  v.dattn = (float*)take(sizeof(float) * s.Q * s.da);
  v.dqv = (float*)take(sizeof(float) * s.Q * s.da);
  v.dKV = (float*)take(sizeof(float) * s.P * 2 * s.da);
  v.tg_part = (float*)take(sizeof(float) * 2 * dtp * gemm_tg_blocks(s.Q));    // query rows
  v.tg_part2 = (float*)take(sizeof(float) * 2 * dtp * gemm_tg_blocks(s.P));   // neighbour slots
  v.S = (float*)take(sizeof(float) * (max_rows > 0 ? max_rows : 1) * W);
  v.head = (float*)take(sizeof(float) * ntiles * W);
  v.tail = (float*)take(sizeof(float) * ntiles * W);
  v.dWkv = (float*)take(sizeof(float) * 2 * s.da * s.Dkv);
  v.dbkv = (float*)take(sizeof(float) * 2 * s.da);
  v.keys = (uint32_t*)take(sizeof(uint32_t) * n_occ);
  v.vals = (uint32_t*)take(sizeof(uint32_t) * n_occ);
  v.seg_lo = (int32_t*)take(sizeof(int32_t) * (max_rows > 0 ? max_rows : 1));
  v.seg_hi = (int32_t*)take(sizeof(int32_t) * (max_rows > 0 ? max_rows : 1));
  v.row_of = (int32_t*)take(sizeof(int32_t) * s.N);
  size_t sc = 0;
  auto mx = [&](size_t x) { if (x > sc) sc = x; };
  {
    // the query weight's problem spans d_m columns when its time columns are closed-form, else D_q;
    // with the query layer on its own (merge_dw_apart) the other three have a region of their own
    const int64_t Ns[4] = {s.da, s.da, s.da, s.da}, Ks[4] = {s.da, s.da + s.dm, s.da, s.Dq};
    const int64_t Ks2[4] = {s.da, s.da + s.dm, s.da, s.dm};
    mx(linear_dw_batch_ws_bytes(s.Q, Ns, Ks, 4));
    mx(linear_dw_batch_ws_bytes(s.Q, Ns, Ks2, 4));
    v.scratch_merge_bytes = 256;
    if (merge_dw_apart(s.Q)) {
      mx(linear_dw_batch_ws_bytes(s.Q, Ns + 3, Ks + 3, 1));
      mx(linear_dw_batch_ws_bytes(s.Q, Ns + 3, Ks2 + 3, 1));
      v.scratch_merge_bytes = a256(linear_dw_batch_ws_bytes(s.Q, Ns, Ks, 3));
    }
    v.scratch_merge = take(v.scratch_merge_bytes);
  }
  mx(linear_dw_ws_bytes(s.P, 2 * s.da, s.Dkv));
  v.scratch = take(sc > 0 ? sc : 1);
  v.scratch_bytes = a256(sc > 0 ? sc : 1);
  v.sort_scratch_bytes = a256(radix_sort_ws_bytes(n_occ));
  v.sort_scratch = take(v.sort_scratch_bytes);
  v.total = (size_t)(w - (char*)base);
  return v;
}

__global__ void k_seg_clear(int32_t* __restrict__ seg_lo, int32_t* __restrict__ seg_hi, int64_t n) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r < n) seg_lo[r] = seg_hi[r] = 0;
}

}  // namespace

size_t segsum_rows_ws_bytes(int64_t n_occ, int64_t max_rows, int dm) {
  const int64_t nt = cdiv(n_occ < 1 ? 1 : n_occ, SEG_TILE_ROWS), mr = max_rows < 1 ? 1 : max_rows;
  return 2 * a256(sizeof(int32_t) * mr) + 2 * a256(sizeof(float) * nt * dm);
}

mtgnn_status segsum_rows(const uint32_t* skeys, const uint32_t* svals, int64_t n_occ, const float* src, int64_t ld,
                         int dm, const int32_t* n_rows, int64_t max_rows, float* D, void* ws, size_t ws_bytes,
                         hipStream_t s) {
  if (dm < 1 || dm > 512) return MTGNN_EUNSUPPORTED;
  if (ws_bytes < segsum_rows_ws_bytes(n_occ, max_rows, dm)) return MTGNN_EWORKSPACE;
  if (max_rows <= 0) return MTGNN_OK;
  const int64_t ntiles = cdiv(n_occ < 1 ? 1 : n_occ, SEG_TILE_ROWS);
  char* w = (char*)ws;
  SegCtx c{};
  c.tile = SEG_TILE_ROWS;
  c.seg_lo = (int32_t*)w;
  w += a256(sizeof(int32_t) * max_rows);
  c.seg_hi = (int32_t*)w;
  w += a256(sizeof(int32_t) * max_rows);
  c.head = (float*)w;
  w += a256(sizeof(float) * ntiles * dm);
  c.tail = (float*)w;
  // every occurrence reads its row from src (all of them are "query" rows; no slot part)
  c.keys = skeys; c.vals = svals; c.n_occ = n_occ; c.sentinel = (uint32_t)max_rows; c.max_q = n_occ;
  c.dhq = src; c.ldq = ld; c.dkv = nullptr; c.dm = dm; c.w2 = 0; c.S = nullptr; c.D = D;
  k_seg_clear<<<(unsigned)cdiv(max_rows, 256), 256, 0, s>>>((int32_t*)c.seg_lo, (int32_t*)c.seg_hi, max_rows);
  MTGNN_CHECK_LAUNCH("seg_clear");
  if (n_occ > 0) {
    k_seg_bounds<<<(unsigned)cdiv(n_occ, 256), 256, 0, s>>>(skeys, n_occ, c.sentinel, (int32_t*)c.seg_lo,
                                                             (int32_t*)c.seg_hi);
    MTGNN_CHECK_LAUNCH("seg_bounds");
    const unsigned gt = (unsigned)cdiv(ntiles, 4);
    if (dm % 4 == 0 && ld % 4 == 0 && ((uintptr_t)src | (uintptr_t)D) % 16 == 0) {
      k_segsum_tiles_v4<<<gt, 256, 0, s>>>(c);
    } else {
      switch (cdiv(dm, 64)) {
        case 1: k_segsum_tiles<1><<<gt, 256, 0, s>>>(c); break;
        case 2: k_segsum_tiles<2><<<gt, 256, 0, s>>>(c); break;
        case 3: k_segsum_tiles<3><<<gt, 256, 0, s>>>(c); break;
        case 4: k_segsum_tiles<4><<<gt, 256, 0, s>>>(c); break;
        case 5: k_segsum_tiles<5><<<gt, 256, 0, s>>>(c); break;
        case 6: k_segsum_tiles<6><<<gt, 256, 0, s>>>(c); break;
        case 7: k_segsum_tiles<7><<<gt, 256, 0, s>>>(c); break;
        default: k_segsum_tiles<8><<<gt, 256, 0, s>>>(c); break;
      }
    }
    MTGNN_CHECK_LAUNCH("segsum_tiles");
  }
  launch_segsum_fixup(c, n_rows, max_rows, n_occ > 0 ? ntiles : 0, s);
  MTGNN_CHECK_LAUNCH("segsum_fixup");
  return MTGNN_OK;
}

size_t attn_save_bytes(const mtgnn_dims* d, int64_t max_q) { return carve_save(nullptr, AttnShape(d, max_q)).total; }

size_t attn_fwd_ws(const mtgnn_dims*, int64_t max_q) { return scan_ws_bytes(max_q); }

mtgnn_status attn_prepare_weights_impl(const mtgnn_attn_params* p, const float* tw, const float* tb,
                                       const mtgnn_dims* d, void* save, hipStream_t s, const PadCopy* more,
                                       int n_more) {
  if (n_more < 0 || n_more > 4) return MTGNN_EINVAL;
  const AttnShape sh(d, 0);
  const AttnSave sv = carve_save(save, sh);
  if (merge_fused_ok(d->dtype, sh.da, sh.dm)) {   // float32: one launch for every copy
    PadCopy ex[12] = {plain_copy((const float*)p->W_k, (float*)sv.W_kv, sh.da, (int)sh.Dkv),
                     plain_copy((const float*)p->W_v, (float*)sv.W_kv + (size_t)sh.da * sh.Dkv, sh.da, (int)sh.Dkv),
                     plain_copy(p->b_k, sv.b_kv, 1, sh.da), plain_copy(p->b_v, sv.b_kv + sh.da, 1, sh.da)};
    int n_ex = 4;
    const bool qf = qproj_fused_ok(d->dtype, sh.da, sh.dm, sh.dt);
    if (qf) {
      ex[n_ex++] = qproj_copy((const float*)p->W_q, sh.da, sh.dm, sh.dt, sv.merge_w, 0);
      ex[n_ex++] = qproj_copy((const float*)p->W_q, sh.da, sh.dm, sh.dt, sv.merge_w, 1);
      for (int which = 0; which < 2; ++which)
        ex[n_ex++] = dmem_copy((const float*)p->W_k, (const float*)p->W_v, sh.da, sh.dm, sh.dt, (int)sh.Dkv,
                               sv.merge_w, which);
    }
    for (int i = 0; i < n_more; ++i) ex[n_ex++] = more[i];
    const QConst qc{(const float*)p->W_q, p->b_q, tw, tb, sv.qc, sh.da, sh.dm, sh.dt};
    return merge_prepare((const float*)p->W_o, (const float*)p->W_1, (const float*)p->W_2, sh.da, sh.dm, sv.merge_w,
                         s, ex, n_ex, qf ? &qc : nullptr);
  }
  const int64_t wkv = (int64_t)sh.da * sh.Dkv;
  if (d->dtype == MTGNN_F32)
    k_stack_kv<float><<<(unsigned)cdiv(wkv, 256), 256, 0, s>>>((const float*)p->W_k, (const float*)p->W_v, p->b_k,
                                                               p->b_v, sh.da, sh.Dkv, (float*)sv.W_kv, sv.b_kv);
  else
    k_stack_kv<uint16_t><<<(unsigned)cdiv(wkv, 256), 256, 0, s>>>((const uint16_t*)p->W_k, (const uint16_t*)p->W_v,
                                                                  p->b_k, p->b_v, sh.da, sh.Dkv,
                                                                  (uint16_t*)sv.W_kv, sv.b_kv);
  MTGNN_CHECK_LAUNCH("stack_kv");
  return pad_copies(more, n_more, s);
}

mtgnn_status attn_prepare_slots_impl(const int32_t* nbr, const int32_t* n_q, int64_t max_q, const mtgnn_dims* d,
                                     void* save, void* ws, size_t ws_bytes, hipStream_t s) {
  const AttnShape sh(d, max_q);
  const AttnSave sv = carve_save(save, sh);
  k_pair_counts<<<(unsigned)cdiv(max_q, 256), 256, 0, s>>>(nbr, n_q, max_q, sh.k, sv.cnt);
  MTGNN_CHECK_LAUNCH("pair_counts");
  return scan_exclusive(sv.cnt, sv.pair_off, max_q, sv.n_valid, ws, ws_bytes, s);
}

mtgnn_status attn_prepare_impl(const int32_t* nbr, const int32_t* n_q, int64_t max_q, const mtgnn_attn_params* p,
                               const float* tw, const float* tb, const mtgnn_dims* d, void* save, void* ws,
                               size_t ws_bytes, hipStream_t s) {
  MTGNN_TRY(attn_prepare_weights_impl(p, tw, tb, d, save, s));
  return attn_prepare_slots_impl(nbr, n_q, max_q, d, save, ws, ws_bytes, s);
}

mtgnn_status attn_fwd_impl(const int32_t* q_node, const float* q_t, const int32_t* n_q, int64_t max_q,
                           const int32_t* nbr, const float* nt, const int32_t* neid, const void* memory,
                           const float* edge_feat, const float* tw, const float* tb, const mtgnn_attn_params* p,
                           const mtgnn_dims* d, float* z, void* save, void* ws, size_t ws_bytes, hipStream_t s) {
  MTGNN_TRY(attn_prepare_impl(nbr, n_q, max_q, p, tw, tb, d, save, ws, ws_bytes, s));
  return attn_fwd_prepared_impl(q_node, q_t, n_q, max_q, nbr, nt, neid, memory, edge_feat, tw, tb, p, d, z, save, s);
}

mtgnn_status attn_fwd_prepared_impl(const int32_t* q_node, const float* q_t, const int32_t* n_q, int64_t max_q,
                                    const int32_t* nbr, const float* nt, const int32_t* neid, const void* memory,
                                    const float* edge_feat, const float* tw, const float* tb,
                                    const mtgnn_attn_params* p, const mtgnn_dims* d, float* z, void* save,
                                    hipStream_t s) {
  const AttnShape sh(d, max_q);
  const AttnSave sv = carve_save(save, sh);
  const int bf = d->dtype == MTGNN_BF16 ? 1 : 0;
  const int wt = d->dtype;
  const unsigned gq = (unsigned)cdiv(sh.Q, 4);
  const GatherArgs ga{q_node, nbr, neid, n_q, sv.cnt, sv.pair_off, nt, q_t, edge_feat, tw, tb, max_q, sh.k, sh.dm,
                      sh.de, sh.dt, sh.da, bf, sv.q_in, sv.m_in, sv.kv_in, sv.pair_delta, sv.pair_nbr};
  const bool v4 = sh.de % 4 == 0 && sh.dm % 4 == 0 && sh.dt % 4 == 0 && sh.da % 4 == 0 && sh.dt <= GV_MAX_DT &&
                  ((uintptr_t)memory & (bf ? 7 : 15)) == 0 && (sh.de == 0 || ((uintptr_t)edge_feat & 15) == 0);
  if (v4 && !bf)
    k_attn_gather_v4<float><<<gq, 256, 0, s>>>(ga, (const float*)memory);
  else if (v4)
    k_attn_gather_v4<uint16_t><<<gq, 256, 0, s>>>(ga, (const uint16_t*)memory);
  else if (!bf)
    k_attn_gather<float><<<gq, 256, 0, s>>>(ga, (const float*)memory);
  else
    k_attn_gather<uint16_t><<<gq, 256, 0, s>>>(ga, (const uint16_t*)memory);
  MTGNN_CHECK_LAUNCH("attn_gather");
  if (qproj_fused_ok(d->dtype, sh.da, sh.dm, sh.dt))
    MTGNN_TRY(qproj_fwd_fused(sv.q_in, sv.merge_w, sv.qc, sv.qv, n_q, max_q, sh.da, sh.dm, sh.dt, s));
  else
    MTGNN_TRY(linear_fwd(sv.q_in, MTGNN_F32, sh.Dq, p->W_q, wt, sh.Dq, p->b_q, sv.qv, sh.da, sh.Q, n_q, sh.da, sh.Dq,
                         false, s));
  MTGNN_TRY(linear_fwd<site::KvProj>(sv.kv_in, MTGNN_F32, sh.Dkv, sv.W_kv, wt, sh.Dkv, sv.b_kv, sv.KV, 2 * sh.da,
                                     sh.P, sv.n_valid, 2 * sh.da, sh.Dkv, false, s));
  {
    TimedScope ts("k_attn_core", s);
    const bool v4 = sh.da % 4 == 0 && sh.da <= 128 && sh.H <= 2 && sh.k <= 20;
    if (v4 && sh.k <= 10 && sh.H == 2)
      k_attn_core_v4<5, 2><<<gq, 256, 0, s>>>(sv.qv, sv.KV, sv.cnt, sv.pair_off, n_q, max_q, sh.k, sh.da, bf, sv.p,
                                              sv.attn);
    else if (v4 && sh.H == 2)
      k_attn_core_v4<10, 2><<<gq, 256, 0, s>>>(sv.qv, sv.KV, sv.cnt, sv.pair_off, n_q, max_q, sh.k, sh.da, bf, sv.p,
                                               sv.attn);
    else if (v4 && sh.k <= 10)
      k_attn_core_v4<5, 1><<<gq, 256, 0, s>>>(sv.qv, sv.KV, sv.cnt, sv.pair_off, n_q, max_q, sh.k, sh.da, bf, sv.p,
                                              sv.attn);
    else if (v4)
      k_attn_core_v4<10, 1><<<gq, 256, 0, s>>>(sv.qv, sv.KV, sv.cnt, sv.pair_off, n_q, max_q, sh.k, sh.da, bf, sv.p,
                                               sv.attn);
    else if (sh.dh <= 64)
      k_attn_core<1><<<gq, 256, 0, s>>>(sv.qv, sv.KV, sv.cnt, sv.pair_off, n_q, max_q, sh.k, sh.da, sh.H, bf, sv.p,
                                        sv.attn);
    else
      k_attn_core<MAX_DH_CHUNKS><<<gq, 256, 0, s>>>(sv.qv, sv.KV, sv.cnt, sv.pair_off, n_q, max_q, sh.k, sh.da, sh.H,
                                                    bf, sv.p, sv.attn);
  }
  MTGNN_CHECK_LAUNCH("attn_core");
  const int64_t ldm = sh.da + sh.dm;
  if (merge_fused_ok(d->dtype, sh.da, sh.dm)) {
    return merge_fwd_fused(sv.attn, sv.m_in, sv.merge_w, p->b_o, p->b_1, p->b_2, sv.m1, sv.a1, z, n_q, max_q, sh.da,
                           sh.dm, s);
  }
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

namespace {

// d M' for the updated rows (reads dh_q in dm_in[:, da:], dK|dV, the slot nodes and
// [W_k; W_v]; writes d_mem).  Its workspace regions (keys, vals, segment bounds, row
// map, S, tile partials, sort scratch) are disjoint from the parameter part's.
// d M' grouping, first half: every occurrence (query rows, then compact neighbour slots) keyed by
// the updated row of its node (or the sentinel max_rows), sorted stably by key, and each row's
// segment bounds.  Reads only forward outputs and the updated-row list, so it may run before
// any gradient exists.  *skeys / *svals: the buffers holding the sorted pairs.
mtgnn_status attn_bwd_dmem_group(const int32_t* q_node, const int32_t* n_q, int64_t max_q, const int32_t* nbr,
                                 const AttnShape& sh, const AttnSave& sv, const BwdWs& b, const int32_t* uniq,
                                 const int32_t* n_rows, int64_t max_rows, uint32_t** skeys, uint32_t** svals,
                                 hipStream_t s) {
  const int64_t n_occ = sh.Q + sh.P;
  const uint32_t sentinel = (uint32_t)max_rows;
  k_row_map<<<(unsigned)cdiv(max_rows, 256), 256, 0, s>>>(uniq, n_rows, max_rows, b.row_of, b.seg_lo, b.seg_hi);
  MTGNN_CHECK_LAUNCH("row_map");
  k_occ_keys<<<(unsigned)cdiv(n_occ, 256), 256, 0, s>>>(q_node, nbr, sv.cnt, sv.pair_off, n_q, max_q, sh.k,
                                                         sv.n_valid, sh.P, uniq, n_rows, max_rows, b.row_of, sentinel,
                                                         b.keys, b.vals);
  MTGNN_CHECK_LAUNCH("occ_keys");
  *skeys = b.keys;
  *svals = b.vals;
  MTGNN_TRY(radix_sort_pairs(skeys, svals, n_occ, bits_for(max_rows), b.sort_scratch, b.sort_scratch_bytes, s));
  k_seg_bounds<<<(unsigned)cdiv(n_occ, 256), 256, 0, s>>>(*skeys, n_occ, sentinel, b.seg_lo, b.seg_hi);
  MTGNN_CHECK_LAUNCH("seg_bounds");
  return MTGNN_OK;
}

// d M' grouping, second half: per-row sums of [dh_q | dK | dV] over the sorted occurrences, in a
// fixed order, then d M' = (sum of dh_q) + (sum of dK|dV) W_kv[:, :dm].
mtgnn_status attn_bwd_dmem_sum(int64_t max_q, const AttnShape& sh, const AttnSave& sv, const BwdWs& b,
                               const uint32_t* skeys, const uint32_t* svals, const int32_t* n_rows, int64_t max_rows,
                               int wt, float* d_mem, hipStream_t s) {
  const int64_t Q = sh.Q, P = sh.P, ldm = sh.da + sh.dm;
  const int da = sh.da, dm = sh.dm;
  {
    const int64_t n_occ = Q + P;
    const uint32_t sentinel = (uint32_t)max_rows;
    SegCtx c;
    c.keys = (uint32_t*)skeys; c.vals = (uint32_t*)svals; c.n_occ = n_occ; c.sentinel = sentinel; c.max_q = max_q;
    c.seg_lo = b.seg_lo; c.seg_hi = b.seg_hi;
    c.dhq = b.dm_in + da; c.ldq = ldm; c.dkv = b.dKV; c.dm = dm; c.w2 = 2 * da;
    c.S = b.S; c.D = d_mem; c.head = b.head; c.tail = b.tail; c.tile = SEG_TILE;
    const int64_t ntiles = cdiv(n_occ, SEG_TILE);
    const unsigned gt = (unsigned)cdiv(ntiles, 4);
    if (dm % 4 == 0 && da % 4 == 0 && dm + 2 * da <= 512) {   // 16-byte aligned rows and groups
      k_segsum_tiles_v4<<<gt, 256, 0, s>>>(c);
    } else {
      switch (cdiv(dm + 2 * da, 64)) {   // column chunks per lane (validation keeps the width <= 512)
        case 1: k_segsum_tiles<1><<<gt, 256, 0, s>>>(c); break;
        case 2: k_segsum_tiles<2><<<gt, 256, 0, s>>>(c); break;
        case 3: k_segsum_tiles<3><<<gt, 256, 0, s>>>(c); break;
        case 4: k_segsum_tiles<4><<<gt, 256, 0, s>>>(c); break;
        case 5: k_segsum_tiles<5><<<gt, 256, 0, s>>>(c); break;
        case 6: k_segsum_tiles<6><<<gt, 256, 0, s>>>(c); break;
        case 7: k_segsum_tiles<7><<<gt, 256, 0, s>>>(c); break;
        default: k_segsum_tiles<8><<<gt, 256, 0, s>>>(c); break;
      }
    }
    MTGNN_CHECK_LAUNCH("segsum_tiles");
    launch_segsum_fixup(c, n_rows, max_rows, ntiles, s);
    MTGNN_CHECK_LAUNCH("segsum_fixup");
    const int W = dm + 2 * da;
    if (qproj_fused_ok(wt, da, dm, sh.dt))
      MTGNN_TRY(dmem_dx_fused(b.S, W, sv.merge_w, d_mem, n_rows, max_rows, da, dm, sh.dt, s));
    else
      MTGNN_TRY(linear_dx(b.S + dm, W, sv.W_kv, wt, sh.Dkv, d_mem, dm, max_rows, n_rows, 2 * da, dm, true, s));
  }
  return MTGNN_OK;
}

// Weight gradients of the merge MLP and the output projection, one batch over the query rows: they need
// only dz and the merge backward's dm1 and do (dm_in's first d_a columns), so with a second stream they
// run there while the score backward and the query projection's data gradient run on `stream`.
mtgnn_status attn_bwd_merge_dw(const int32_t* n_q, const AttnShape& sh, const AttnSave& sv, const BwdWs& b,
                               const float* dz, mtgnn_attn_grads* g, hipStream_t s) {
  const int64_t ldm = sh.da + sh.dm;
  const int da = sh.da;
  const DwProblem ps[3] = {{dz, da, sv.a1, da, g->W_2, da, da, da, g->b_2},
                           {b.dm1, da, sv.m_in, ldm, g->W_1, ldm, da, ldm, g->b_1},
                           {b.dm_in, ldm, sv.attn, da, g->W_o, da, da, da, g->b_o}};
  return linear_dw_batch(ps, 3, sh.Q, n_q, MTGNN_F32, b.scratch_merge, b.scratch_merge_bytes, s);
}

// The parameter gradients that follow the fork point (weight gradient of the
// query layer and of [W_k; W_v], the time-encoder gradients).
mtgnn_status attn_bwd_params(const int32_t* n_q, const AttnShape& sh, const AttnSave& sv, const BwdWs& b,
                             const float* dz, const float* tw, const float* tb, const mtgnn_attn_params* p,
                             int wt, mtgnn_attn_grads* g, float* d_time_w, float* d_time_b, hipStream_t s) {
  const int64_t Q = sh.Q, P = sh.P;
  const int da = sh.da, dm = sh.dm, dt = sh.dt;
  char* sc = b.scratch;
  const size_t scb = b.scratch_bytes;
  auto wofs = [&](const void* W, int64_t col) { return (const void*)((const char*)W + sh.esz * (size_t)col); };
  // Order: the time-encoder gradients and the data-gradient product first, the
  // weight gradients last, so that the d M' part (on its own stream when
  // overlapped) shares the GPU with the smaller products rather than with the
  // key/value weight gradient.
  // Time-encoder gradient: phi(tau - t_j) of the neighbour slots (sin(arg) recomputed in the
  // product's epilogue from the saved tau - t_j), and phi(0) of the queries.  In float32 the queries' share is closed-form from the query projection's bias
  // gradient (their delta is 0), added in the reduce after the weight-gradient batch; otherwise it
  // is a product of its own (its w part is zero, its b part is not).
  const bool q_closed = wt == MTGNN_F32;
  if (dt > 0) {
    if (!q_closed)
      MTGNN_TRY(linear_dx_timegrad(b.dqv, da, wofs(p->W_q, dm), wt, sh.Dq, Q, n_q, da, dt, nullptr, nullptr, tw, tb,
                                   b.tg_part, s));
    MTGNN_TRY(linear_dx_timegrad<site::KvDx>(b.dKV, 2 * da, wofs(sv.W_kv, dm + sh.de), wt, sh.Dkv, P, sv.n_valid,
                                             2 * da, dt, nullptr, sv.pair_delta, tw, tb, b.tg_part2, s));
    if (!q_closed)
      MTGNN_TRY(timegrad_reduce_blocks2(b.tg_part, Q, n_q, b.tg_part2, P, sv.n_valid, G_TG_ROWS, dt, d_time_w,
                                        d_time_b, s));
  }
  // weight gradients of the query, output and merge layers, one batch over the query rows (the query
  // layer's alone when the others run apart: attn_bwd_merge_dw)
  {
    const int64_t ldm = sh.da + sh.dm;
    const DwProblem ps[4] = {{dz, da, sv.a1, da, g->W_2, da, da, da, g->b_2},
                             {b.dm1, da, sv.m_in, ldm, g->W_1, ldm, da, ldm, g->b_1},
                             {b.dm_in, ldm, sv.attn, da, g->W_o, da, da, da, g->b_o},
                             {b.dqv, da, sv.q_in, sh.Dq, g->W_q, sh.Dq, da, q_closed && dt > 0 ? dm : sh.Dq, g->b_q}};
    if (merge_dw_apart(Q)) MTGNN_TRY(linear_dw_batch(ps + 3, 1, Q, n_q, MTGNN_F32, sc, scb, s));
    else MTGNN_TRY(linear_dw_batch(ps, 4, Q, n_q, MTGNN_F32, sc, scb, s));
  }
  if (dt > 0 && q_closed)
    MTGNN_TRY(timegrad_reduce_slots_q(b.tg_part2, P, sv.n_valid, G_TG_ROWS, dt, g->b_q, (const float*)p->W_q, sh.Dq,
                                      dm, da, tw, tb, d_time_w, d_time_b, g->W_q, s));
  // key/value projection over the compact slots (stacked [W_k; W_v]); the output-stationary kernel's
  // reduce writes the W_k and W_v halves (rows < d_a, rows >= d_a) straight to their gradients
  if (dw_rs_applicable(b.dKV, 2 * da, 2 * da, sv.kv_in, MTGNN_F32, sh.Dkv, (int)sh.Dkv))
    return dw_rs_launch_rows2(b.dKV, 2 * da, 2 * da, sv.kv_in, sh.Dkv, (int)sh.Dkv, P, sv.n_valid, g->W_k, g->W_v,
                              sh.Dkv, g->b_k, g->b_v, da, sc, scb, s);
  MTGNN_TRY(linear_dw<site::KvDw>(b.dKV, 2 * da, sv.kv_in, MTGNN_F32, sh.Dkv, b.dWkv, sh.Dkv, P, sv.n_valid, 2 * da,
                                  sh.Dkv, sc, scb, s, b.dbkv));
  k_split_kv_grads<<<(unsigned)cdiv((int64_t)da * sh.Dkv, 256), 256, 0, s>>>(b.dWkv, b.dbkv, da, sh.Dkv, g->W_k,
                                                                              g->W_v, g->b_k, g->b_v);
  MTGNN_CHECK_LAUNCH("split_kv_grads");
  return MTGNN_OK;
}

}  // namespace

mtgnn_status attn_bwd_group_impl(const int32_t* q_node, const int32_t* n_q, int64_t max_q, const int32_t* nbr,
                                 const void* save, const int32_t* uniq, const int32_t* n_rows, int64_t max_rows,
                                 const mtgnn_dims* d, void* ws, size_t ws_bytes, hipStream_t s) {
  const AttnShape sh(d, max_q);
  const AttnSave sv = carve_save((void*)save, sh);
  const BwdWs b = carve_bwd(ws, sh, max_rows);
  if (ws_bytes < b.total) return MTGNN_EWORKSPACE;
  if (max_rows == 0) return MTGNN_OK;
  uint32_t *skeys = nullptr, *svals = nullptr;
  return attn_bwd_dmem_group(q_node, n_q, max_q, nbr, sh, sv, b, uniq, n_rows, max_rows, &skeys, &svals, s);
}

mtgnn_status attn_bwd_impl(const int32_t* q_node, const float* q_t, const int32_t* n_q, int64_t max_q,
                           const int32_t* nbr, const float* nt, const float* dz, const void* save, const int32_t* uniq,
                           const int32_t* n_rows, int64_t max_rows, const float* tw, const float* tb,
                           const mtgnn_attn_params* p, const mtgnn_dims* d, mtgnn_attn_grads* g, float* d_mem,
                           float* d_time_w, float* d_time_b, void* ws, size_t ws_bytes, hipStream_t s,
                           hipStream_t s_dmem, hipEvent_t fork, hipEvent_t join, bool grouped) {
  (void)q_t;
  (void)nt;
  const AttnShape sh(d, max_q);
  const AttnSave sv = carve_save((void*)save, sh);
  const BwdWs b = carve_bwd(ws, sh, max_rows);
  if (ws_bytes < b.total) return MTGNN_EWORKSPACE;
  const int wt = d->dtype;
  const int64_t Q = sh.Q, ldm = sh.da + sh.dm;
  const int da = sh.da, dm = sh.dm;

  // With a second stream, the d M' grouping's key sort starts there at once (it reads only forward
  // outputs): first fork.  The same event marks the second fork below.  `grouped`: the grouping is
  // already in ws (attn_bwd_group_impl, ordered before the second stream's next work).
  const bool overlap = s_dmem != nullptr && max_rows > 0;
  uint32_t *skeys = nullptr, *svals = nullptr;
  if (overlap && grouped) {
    skeys = b.keys;
    svals = b.vals;
    radix_sort_output(&skeys, &svals, sh.Q + sh.P, bits_for(max_rows), b.sort_scratch);
  } else if (overlap) {
    hipError_t e0 = hipEventRecord(fork, s);
    if (e0 == hipSuccess) e0 = hipStreamWaitEvent(s_dmem, fork, 0);
    if (e0 != hipSuccess) {
      set_hip_error(e0, "attn_bwd fork");
      return MTGNN_EHIP;
    }
    const mtgnn_status st0 =
        attn_bwd_dmem_group(q_node, n_q, max_q, nbr, sh, sv, b, uniq, n_rows, max_rows, &skeys, &svals, s_dmem);
    if (st0 != MTGNN_OK) {   // leave `stream` ordered after the second stream
      if (hipEventRecord(join, s_dmem) == hipSuccess) (void)hipStreamWaitEvent(s, join, 0);
      return st0;
    }
  }
  // data gradients down to dK|dV and dh_q, on `stream`
  auto chain = [&]() -> mtgnn_status {
    // merge MLP: z = W_2 a1 + b_2, a1 = relu(m1), m1 = W_1 m_in + b_1
    // (their weight gradients run as one batch after the score backward)
    // output projection: o = W_o attn + b_o   (do = dm_in[:, :da])
    if (merge_fused_ok(wt, da, dm)) {
      MTGNN_TRY(merge_bwd_fused(dz, sv.merge_w, sv.m1, b.dm1, b.dm_in, b.dattn, n_q, max_q, da, dm, s));
    } else {
      MTGNN_TRY(linear_dx(dz, da, p->W_2, wt, da, b.dm1, da, Q, n_q, da, da, false, s, sv.m1, da));
      MTGNN_TRY(linear_dx(b.dm1, da, p->W_1, wt, ldm, b.dm_in, ldm, Q, n_q, da, ldm, false, s));
      MTGNN_TRY(linear_dx(b.dm_in, ldm, p->W_o, wt, da, b.dattn, da, Q, n_q, da, da, false, s));
    }
    // their weight gradients (many query rows): on the second stream (after a fork) while the rest of the
    // chain runs here (the query projection's data gradient writes dm_in's other columns only)
    if (merge_dw_apart(Q) && overlap) {
      hipError_t e = hipEventRecord(fork, s);
      if (e == hipSuccess) e = hipStreamWaitEvent(s_dmem, fork, 0);
      if (e != hipSuccess) {
        set_hip_error(e, "attn_bwd fork");
        return MTGNN_EHIP;
      }
      MTGNN_TRY(attn_bwd_merge_dw(n_q, sh, sv, b, dz, g, s_dmem));
    } else if (merge_dw_apart(Q)) {
      MTGNN_TRY(attn_bwd_merge_dw(n_q, sh, sv, b, dz, g, s));
    }
    // softmax-weighted sum and scores
    {
      TimedScope ts("k_attn_core_bwd", s);
      const bool v4 = sh.da % 4 == 0 && sh.da <= 128 && sh.H <= 2 && sh.k <= 20;
      const unsigned gq = (unsigned)cdiv(Q, 4);
      if (v4 && sh.k <= 10 && sh.H == 2)
        k_attn_core_bwd_v4<5, 2><<<gq, 256, 0, s>>>(sv.qv, sv.KV, sv.p, b.dattn, sv.cnt, sv.pair_off, n_q, max_q,
                                                    sh.k, da, b.dKV, b.dqv);
      else if (v4 && sh.H == 2)
        k_attn_core_bwd_v4<10, 2><<<gq, 256, 0, s>>>(sv.qv, sv.KV, sv.p, b.dattn, sv.cnt, sv.pair_off, n_q, max_q,
                                                     sh.k, da, b.dKV, b.dqv);
      else if (v4 && sh.k <= 10)
        k_attn_core_bwd_v4<5, 1><<<gq, 256, 0, s>>>(sv.qv, sv.KV, sv.p, b.dattn, sv.cnt, sv.pair_off, n_q, max_q,
                                                    sh.k, da, b.dKV, b.dqv);
      else if (v4)
        k_attn_core_bwd_v4<10, 1><<<gq, 256, 0, s>>>(sv.qv, sv.KV, sv.p, b.dattn, sv.cnt, sv.pair_off, n_q, max_q,
                                                     sh.k, da, b.dKV, b.dqv);
      else if (sh.dh <= 64)
        k_attn_core_bwd<1><<<(unsigned)cdiv(Q, 4), 256, 0, s>>>(sv.qv, sv.KV, sv.p, b.dattn, sv.cnt, sv.pair_off,
                                                                 n_q, max_q, sh.k, da, sh.H, b.dKV, b.dqv);
      else
        k_attn_core_bwd<MAX_DH_CHUNKS><<<(unsigned)cdiv(Q, 4), 256, 0, s>>>(sv.qv, sv.KV, sv.p, b.dattn, sv.cnt,
                                                                             sv.pair_off, n_q, max_q, sh.k, da, sh.H,
                                                                             b.dKV, b.dqv);
    }
    MTGNN_CHECK_LAUNCH("attn_core_bwd");
    // query projection, data gradient: dhq += dqv W_q[:, :dm] (the last input of the d M' grouping)
    if (qproj_fused_ok(wt, da, dm, sh.dt))
      MTGNN_TRY(qproj_dx_fused(b.dqv, sv.merge_w, b.dm_in, ldm, n_q, max_q, da, dm, sh.dt, s));
    else
      MTGNN_TRY(linear_dx(b.dqv, da, p->W_q, wt, sh.Dq, b.dm_in + da, ldm, Q, n_q, da, dm, true, s));
    return MTGNN_OK;
  };
  if (const mtgnn_status st1 = chain(); st1 != MTGNN_OK) {
    if (overlap && join && hipEventRecord(join, s_dmem) == hipSuccess) (void)hipStreamWaitEvent(s, join, 0);
    return st1;
  }
  if (!overlap) {
    MTGNN_TRY(attn_bwd_params(n_q, sh, sv, b, dz, tw, tb, p, wt, g, d_time_w, d_time_b, s));
    if (max_rows > 0) {
      MTGNN_TRY(attn_bwd_dmem_group(q_node, n_q, max_q, nbr, sh, sv, b, uniq, n_rows, max_rows, &skeys, &svals, s));
      MTGNN_TRY(attn_bwd_dmem_sum(max_q, sh, sv, b, skeys, svals, n_rows, max_rows, wt, d_mem, s));
    }
    return MTGNN_OK;
  }
  // second fork: the sums of d M' on the second stream, the parameter gradients here; join before returning
  // (join == NULL, grouped form only: the caller orders `stream` after the second stream itself)
  hipError_t e = hipEventRecord(fork, s);
  if (e == hipSuccess) e = hipStreamWaitEvent(s_dmem, fork, 0);
  if (e != hipSuccess) {
    set_hip_error(e, "attn_bwd fork");
    return MTGNN_EHIP;
  }
  MTGNN_TRY(attn_bwd_dmem_sum(max_q, sh, sv, b, skeys, svals, n_rows, max_rows, wt, d_mem, s_dmem));
  if (!join) return attn_bwd_params(n_q, sh, sv, b, dz, tw, tb, p, wt, g, d_time_w, d_time_b, s);
  e = hipEventRecord(join, s_dmem);
  if (e != hipSuccess) {
    set_hip_error(e, "attn_bwd join");
    return MTGNN_EHIP;
  }
  const mtgnn_status st = attn_bwd_params(n_q, sh, sv, b, dz, tw, tb, p, wt, g, d_time_w, d_time_b, s);
  e = hipStreamWaitEvent(s, join, 0);   // even after a failure, leave `stream` ordered after the second stream
  if (e != hipSuccess) {
    set_hip_error(e, "attn_bwd join wait");
    return MTGNN_EHIP;
  }
  return st;
}

}  // namespace mtgnn

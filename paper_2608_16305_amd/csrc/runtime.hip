// Adaptive runtime controller of one worker (Section V, Algorithm 2): the host-side decision state
// (Eq. 6-9), and the device work around a batch step: PruneAux (Eq. 10-11), the boundary cache refresh
// (Eq. 25), the gradient norm g_r that drives the synchronization decision, and the parameter update.
#include <cmath>
#include <new>

#include "ops.h"

struct mtgnn_controller {
  mtgnn_controller_config cfg;
  double g_bar = 0, g_last = 0, c_bar = 0, c_prev = 0;
};

namespace mtgnn {

namespace {

// ---------------------------------------------------------------- gradient norm

constexpr int GN_CHUNK = 4096;   // elements per block

struct GradSet {
  const float* p[RT_MAX_TENSORS];
  int64_t n[RT_MAX_TENSORS];
  int64_t first_block[RT_MAX_TENSORS + 1];
  int count;
};

// Sum of squares of one chunk of one tensor, in double, in a fixed order (256 threads, then a fixed tree).
__global__ __launch_bounds__(256) void k_sumsq_partial(GradSet g, double* __restrict__ part) {
  __shared__ double red[256];
  const int64_t b = blockIdx.x;
  int i = 0;
  while (i + 1 < g.count && g.first_block[i + 1] <= b) ++i;
  const int64_t lo = (b - g.first_block[i]) * GN_CHUNK;
  const int64_t hi = min(g.n[i], lo + GN_CHUNK);
  double s = 0.0;
  for (int64_t e = lo + threadIdx.x; e < hi; e += 256) {
    const double v = g.p[i][e];
    s += v * v;
  }
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) part[b] = red[0];
}

__global__ __launch_bounds__(256) void k_sumsq_final(const double* __restrict__ part, int64_t n_part,
                                                     double* __restrict__ norm) {
  __shared__ double red[256];
  double s = 0.0;
  for (int64_t b = threadIdx.x; b < n_part; b += 256) s += part[b];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) *norm = sqrt(red[0]);
}

// ---------------------------------------------------------------- PruneAux

__global__ void k_prune_aux(uint8_t* __restrict__ flags, int64_t n, int heavy) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= n) return;
  const uint8_t f = flags[e];
  flags[e] = ((f & 1) && heavy) ? (uint8_t)(f | 2) : (uint8_t)(f & ~2);
}

// ---------------------------------------------------------------- cache refresh

// A wave per 32-node word of the refresh set: every set bit's memory row and last update time are
// copied from the authoritative table (rows of row_bytes bytes, 4-byte multiples).
__global__ __launch_bounds__(256) void k_cache_refresh(const uint32_t* __restrict__ bits, int64_t words,
                                                       int64_t n_nodes, const uint32_t* __restrict__ auth,
                                                       const float* __restrict__ auth_lu, int row_words,
                                                       uint32_t* __restrict__ mem, float* __restrict__ lu) {
  const int64_t w = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (w >= words) return;
  uint32_t m = bits[w];
  while (m) {
    const int b = __ffs(m) - 1;
    m &= m - 1;
    const int64_t node = w * 32 + b;
    if (node >= n_nodes) break;
    for (int c = lane; c < row_words; c += 64) mem[node * row_words + c] = auth[node * row_words + c];
    if (lane == 0) lu[node] = auth_lu[node];
  }
}

// ---------------------------------------------------------------- Adam

struct AdamSet {
  float* p[RT_MAX_TENSORS];
  const float* g[RT_MAX_TENSORS];
  float* m[RT_MAX_TENSORS];
  float* v[RT_MAX_TENSORS];
  uint16_t* shadow[RT_MAX_TENSORS];   // bf16 copy of the parameter, or null
  int64_t n[RT_MAX_TENSORS];
  int64_t first_block[RT_MAX_TENSORS + 1];
  int count;
};

__global__ __launch_bounds__(256) void k_adam(AdamSet a, float lr, float b1, float omb1, float b2, float omb2,
                                              float eps, float bc1, float bc2) {
  const int64_t b = blockIdx.x;
  int i = 0;
  while (i + 1 < a.count && a.first_block[i + 1] <= b) ++i;
  const int64_t e = (b - a.first_block[i]) * 256 + threadIdx.x;
  if (e >= a.n[i]) return;
  const float g = a.g[i][e];
  const float m = b1 * a.m[i][e] + omb1 * g;
  const float v = b2 * a.v[i][e] + omb2 * (g * g);
  a.m[i][e] = m;
  a.v[i][e] = v;
  const float p = a.p[i][e] - lr * (m / bc1) / (sqrtf(v / bc2) + eps);
  a.p[i][e] = p;
  if (a.shadow[i]) a.shadow[i][e] = f32_to_bf16(p);
}

size_t a256r(size_t x) { return (x + 255) & ~size_t(255); }

}  // namespace

size_t grad_norm_ws(const int64_t* sizes, int n) {
  int64_t blocks = 0;
  for (int i = 0; i < n; ++i) blocks += cdiv(sizes[i] < 1 ? 1 : sizes[i], GN_CHUNK);
  return a256r(sizeof(double) * (size_t)(blocks < 1 ? 1 : blocks));
}

mtgnn_status grad_norm_impl(const float* const* grads, const int64_t* sizes, int n, double* norm, void* ws,
                            hipStream_t s) {
  GradSet g{};
  g.count = n;
  int64_t blocks = 0;
  for (int i = 0; i < n; ++i) {
    g.p[i] = grads[i];
    g.n[i] = sizes[i];
    g.first_block[i] = blocks;
    blocks += cdiv(sizes[i] < 1 ? 1 : sizes[i], GN_CHUNK);
  }
  g.first_block[n] = blocks;
  k_sumsq_partial<<<(unsigned)blocks, 256, 0, s>>>(g, (double*)ws);
  MTGNN_CHECK_LAUNCH("sumsq_partial");
  k_sumsq_final<<<1, 256, 0, s>>>((const double*)ws, blocks, norm);
  MTGNN_CHECK_LAUNCH("sumsq_final");
  return MTGNN_OK;
}

mtgnn_status prune_aux_impl(uint8_t* flags, int64_t n, int heavy, hipStream_t s) {
  if (n <= 0) return MTGNN_OK;
  k_prune_aux<<<(unsigned)cdiv(n, 256), 256, 0, s>>>(flags, n, heavy);
  MTGNN_CHECK_LAUNCH("prune_aux");
  return MTGNN_OK;
}

mtgnn_status cache_refresh_impl(const uint32_t* bits, int64_t n_nodes, const void* auth_mem, const float* auth_lu,
                                const mtgnn_dims* d, void* mem, float* lu, hipStream_t s) {
  const int64_t words = cdiv(n_nodes, 32);
  const size_t esz = d->dtype == MTGNN_BF16 ? 2 : 4;
  if ((d->d_mem * esz) % 4 != 0) return MTGNN_EUNSUPPORTED;
  const int row_words = (int)(d->d_mem * esz / 4);
  k_cache_refresh<<<(unsigned)cdiv(words, 4), 256, 0, s>>>(bits, words, n_nodes, (const uint32_t*)auth_mem, auth_lu,
                                                           row_words, (uint32_t*)mem, lu);
  MTGNN_CHECK_LAUNCH("cache_refresh");
  return MTGNN_OK;
}

mtgnn_status adam_impl(float* const* params, const float* const* grads, float* const* m, float* const* v,
                       void* const* shadow, const int64_t* sizes, int n, const mtgnn_adam_config* c,
                       hipStream_t s) {
  AdamSet a{};
  a.count = n;
  int64_t blocks = 0;
  for (int i = 0; i < n; ++i) {
    a.p[i] = params[i];
    a.g[i] = grads[i];
    a.m[i] = m[i];
    a.v[i] = v[i];
    a.shadow[i] = shadow ? (uint16_t*)shadow[i] : nullptr;
    a.n[i] = sizes[i];
    a.first_block[i] = blocks;
    blocks += cdiv(sizes[i] < 1 ? 1 : sizes[i], 256);
  }
  a.first_block[n] = blocks;
  const float bc1 = (float)(1.0 - std::pow((double)c->beta1, (double)c->t));
  const float bc2 = (float)(1.0 - std::pow((double)c->beta2, (double)c->t));
  k_adam<<<(unsigned)blocks, 256, 0, s>>>(a, (float)c->lr, (float)c->beta1, (float)(1.0 - c->beta1), (float)c->beta2,
                                          (float)(1.0 - c->beta2), (float)c->eps, bc1, bc2);
  MTGNN_CHECK_LAUNCH("adam");
  return MTGNN_OK;
}

}  // namespace mtgnn

// ---------------------------------------------------------------- host-side controller (Eq. 6-9)

using namespace mtgnn;

extern "C" {

mtgnn_status mtgnn_controller_create(const mtgnn_controller_config* cfg, mtgnn_controller** out) {
  if (!cfg || !out) return MTGNN_EINVAL;
  if (!(cfg->alpha > 0 && cfg->alpha <= 1) || !(cfg->beta > 0 && cfg->beta <= 1) || !(cfg->tau_g > 0) ||
      !(cfg->tau_c > 0) || cfg->interval <= 0)
    return MTGNN_EINVAL;
  mtgnn_controller* c = new (std::nothrow) mtgnn_controller();
  if (!c) return MTGNN_EINVAL;
  c->cfg = *cfg;
  *out = c;
  return MTGNN_OK;
}

void mtgnn_controller_destroy(mtgnn_controller* c) { delete c; }

mtgnn_status mtgnn_controller_decide(const mtgnn_controller* c, int64_t r, int32_t* boundary, int32_t* sync,
                                     int32_t* heavy) {
  if (!c || r < 0) return MTGNN_EINVAL;
  const bool is_boundary = r % c->cfg.interval == 0;
  if (boundary) *boundary = is_boundary ? 1 : 0;
  // Eq. 7: skip the refresh only in a stable phase: g_{r-1} < tau_g times its EMA
  if (sync) *sync = (is_boundary && !(r > 0 && c->g_bar > 0 && c->g_last < c->cfg.tau_g * c->g_bar)) ? 1 : 0;
  // Eq. 9: heavy load when c_{r-1} exceeds tau_c times its EMA
  if (heavy) *heavy = (r > 0 && c->c_bar > 0 && c->c_prev > c->cfg.tau_c * c->c_bar) ? 1 : 0;
  return MTGNN_OK;
}

mtgnn_status mtgnn_controller_observe(mtgnn_controller* c, double grad_norm, double batch_time) {
  if (!c || !std::isfinite(grad_norm) || !std::isfinite(batch_time) || grad_norm < 0 || batch_time < 0)
    return MTGNN_EINVAL;
  // Eq. 6 and Eq. 8: the first observation initialises each average
  c->g_bar = c->g_bar == 0 ? grad_norm : c->cfg.alpha * grad_norm + (1 - c->cfg.alpha) * c->g_bar;
  c->g_last = grad_norm;
  c->c_bar = c->c_bar == 0 ? batch_time : c->cfg.beta * batch_time + (1 - c->cfg.beta) * c->c_bar;
  c->c_prev = batch_time;
  return MTGNN_OK;
}

mtgnn_status mtgnn_controller_state(const mtgnn_controller* c, double* g_bar, double* g_last, double* c_bar,
                                    double* c_prev) {
  if (!c) return MTGNN_EINVAL;
  if (g_bar) *g_bar = c->g_bar;
  if (g_last) *g_last = c->g_last;
  if (c_bar) *c_bar = c->c_bar;
  if (c_prev) *c_prev = c->c_prev;
  return MTGNN_OK;
}

}  // extern "C"

// Link-prediction decoder and the masked batch loss (Eq. 12-13) with its gradient.
//
// The queries of a batch are the src of its target events, then their dst, then their negatives
// (n_tar rows each, n_tar = n_q / 3 on the device).  An edge (a, b) scores
//   s(a, b) = W_d2 relu(W_d1 [z_a || z_b] + b_d1) + b_d2,
// and the batch loss is the mean over target events of softplus(-s(src, dst)) + softplus(s(src, neg)),
// the binary cross-entropy of the true edge (label 1) and the negative edge (label 0).
//
// W_d1 [z_a || z_b] = W_a z_a + W_b z_b with W_a, W_b the two column halves of W_d1, so the first
// layer is one batched product over all query rows (z W_a^T and z W_b^T); a wave per target event then
// forms both edges' hidden rows, scores, loss terms and hidden-row gradients.  The gradient rows go to
// two query-layout buffers, DA (the src rows: dh_pos + dh_neg; zero elsewhere) and DB (dst rows dh_pos,
// neg rows dh_neg; zero on src rows), so that every remaining product runs over all query rows with
// host-known strides: dz = DA W_a + DB W_b, dW_a = DA^T z, dW_b = DB^T z, db_d1 = column sums of DA.
#include "gemm.h"
#include "ops.h"

namespace mtgnn {

namespace {

size_t al256(size_t x) { return (x + 255) & ~size_t(255); }

__device__ __forceinline__ float softplusf_(float x) { return fmaxf(x, 0.f) + log1pf(expf(-fabsf(x))); }

constexpr int LINK_MAX_COLS = 2;   // columns per lane: d_attn <= 128

// Y [max_q, 2 da]: columns [0, da) = z W_a^T, [da, 2 da) = z W_b^T.  Per target event i (a wave):
// pre_pos = Y[i, :da] + Y[n + i, da:] + b1, pre_neg = Y[i, :da] + Y[2n + i, da:] + b1.
// Hp [max_tar, da + 2]: ds_pos h_pos + ds_neg h_neg | ds_pos + ds_neg | loss term / n (column sums give
// W_d2's and b_d2's gradients and the loss).
__global__ __launch_bounds__(256) void k_link_pairs(const float* __restrict__ Y, const int32_t* __restrict__ n_q,
                                                    int64_t max_tar, int da, const float* __restrict__ b1,
                                                    const float* __restrict__ W2, const float* __restrict__ b2,
                                                    float* __restrict__ DA, float* __restrict__ DB,
                                                    float* __restrict__ Hp, int32_t* __restrict__ n_tar_out,
                                                    float* __restrict__ scores) {
  const int64_t n = (n_q ? (int64_t)*n_q : 3 * max_tar) / 3;
  if (blockIdx.x == 0 && threadIdx.x == 0) *n_tar_out = (int32_t)n;
  const int64_t i = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (i >= n) return;
  const int64_t ld = 2 * da;
  float pp[LINK_MAX_COLS], pn[LINK_MAX_COLS], w2[LINK_MAX_COLS];
  float sp = 0.f, sn = 0.f;
#pragma unroll
  for (int u = 0; u < LINK_MAX_COLS; ++u) {
    const int c = lane + 64 * u;
    pp[u] = pn[u] = w2[u] = 0.f;
    if (c < da) {
      const float a = Y[i * ld + c];
      pp[u] = (a + Y[(n + i) * ld + da + c]) + b1[c];
      pn[u] = (a + Y[(2 * n + i) * ld + da + c]) + b1[c];
      w2[u] = W2[c];
      sp += w2[u] * fmaxf(pp[u], 0.f);
      sn += w2[u] * fmaxf(pn[u], 0.f);
    }
  }
  sp = wave_sum(sp) + b2[0];
  sn = wave_sum(sn) + b2[0];
  const float inv_n = 1.0f / (float)n;
  const float ds_p = (1.0f / (1.0f + expf(-sp)) - 1.0f) * inv_n;   // (sigmoid(s) - 1) / n
  const float ds_n = (1.0f / (1.0f + expf(-sn))) * inv_n;          // sigmoid(s) / n
#pragma unroll
  for (int u = 0; u < LINK_MAX_COLS; ++u) {
    const int c = lane + 64 * u;
    if (c < da) {
      const float dhp = pp[u] > 0.f ? ds_p * w2[u] : 0.f;
      const float dhn = pn[u] > 0.f ? ds_n * w2[u] : 0.f;
      DA[i * da + c] = dhp + dhn;
      DA[(n + i) * da + c] = 0.f;
      DA[(2 * n + i) * da + c] = 0.f;
      DB[i * da + c] = 0.f;
      DB[(n + i) * da + c] = dhp;
      DB[(2 * n + i) * da + c] = dhn;
      Hp[i * (da + 2) + c] = ds_p * fmaxf(pp[u], 0.f) + ds_n * fmaxf(pn[u], 0.f);
    }
  }
  if (lane == 0) {
    Hp[i * (da + 2) + da] = ds_p + ds_n;
    Hp[i * (da + 2) + da + 1] = (softplusf_(-sp) + softplusf_(sn)) * inv_n;
    if (scores) {
      scores[i] = sp;
      scores[max_tar + i] = sn;
    }
  }
}

// sums [da + 2] -> dW_d2 [da], db_d2, loss.
__global__ void k_link_finish(const float* __restrict__ sums, int da, float* __restrict__ dW2,
                              float* __restrict__ db2, float* __restrict__ loss) {
  const int c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c < da) dW2[c] = sums[c];
  if (c == da) db2[0] = sums[da];
  if (c == da + 1) loss[0] = sums[da + 1];
}

struct LinkWs {
  int32_t* n_tar;
  float *Y, *DA, *DB, *Hp, *sums, *db_scratch, *Wp, *part;
  void* rest;
  size_t rest_bytes;
};

size_t link_rest_bytes(int da, int64_t max_q) {
  const int64_t max_tar = max_q / 3;
  const int64_t Ns[2] = {da, da}, Ks[2] = {da, da};
  return std::max(colsum_ws_bytes(max_tar, da + 2), linear_dw_batch_ws_bytes(max_q, Ns, Ks, 2));
}

LinkWs link_ws_layout(void* ws, int da, int64_t max_q, size_t* total = nullptr) {
  const int64_t max_tar = max_q / 3;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += al256(bytes);
    return (char*)ws + o;
  };
  LinkWs L{};
  L.n_tar = (int32_t*)take(sizeof(int32_t));
  L.Y = (float*)take(sizeof(float) * (size_t)max_q * 2 * da);
  L.DA = (float*)take(sizeof(float) * (size_t)max_q * da);
  L.DB = (float*)take(sizeof(float) * (size_t)max_q * da);
  L.Hp = (float*)take(sizeof(float) * (size_t)(max_tar < 1 ? 1 : max_tar) * (da + 2));
  L.sums = (float*)take(sizeof(float) * (size_t)(da + 2));
  L.db_scratch = (float*)take(sizeof(float) * (size_t)da);
  L.Wp = (float*)take(sizeof(float) * link_fused_weight_floats(da));
  L.part = (float*)take(sizeof(float) * (size_t)cdiv(max_tar < 1 ? 1 : max_tar, 16) * (da + 2));
  L.rest_bytes = link_rest_bytes(da, max_q);
  L.rest = take(L.rest_bytes);
  if (total) *total = off;
  return L;
}

}  // namespace

size_t link_loss_ws(const mtgnn_dims* d, int64_t max_q) {
  size_t total = 0;
  char base[1];
  (void)link_ws_layout(base, d->d_attn, max_q, &total);
  return total;
}

int link_copies_impl(const mtgnn_link_params* p, const mtgnn_dims* d, int64_t max_q, void* ws, PadCopy* out) {
  const int da = d->d_attn;
  if (!link_fused_ok(da)) return 0;   // the general widths read W_d1 directly
  const LinkWs L = link_ws_layout(ws, da, max_q);
  return link_pad_copies(p->W_d1, da, L.Wp, out);
}

mtgnn_status link_prepare_impl(const mtgnn_link_params* p, const mtgnn_dims* d, int64_t max_q, void* ws,
                               hipStream_t s) {
  PadCopy c[4];
  const int n = link_copies_impl(p, d, max_q, ws, c);
  return pad_copies(c, n, s);
}

mtgnn_status link_loss_impl(const float* z, const int32_t* n_q, int64_t max_q, const mtgnn_link_params* p,
                            const mtgnn_dims* d, float* loss, float* scores, float* dz, mtgnn_link_grads* g, void* ws,
                            size_t ws_bytes, hipStream_t s, hipStream_t s_dw, hipEvent_t fork, bool prepared) {
  const int da = d->d_attn;
  if (da > 64 * LINK_MAX_COLS) return MTGNN_EUNSUPPORTED;
  if (ws_bytes < link_loss_ws(d, max_q)) return MTGNN_EWORKSPACE;
  const int64_t max_tar = max_q / 3;
  LinkWs L = link_ws_layout(ws, da, max_q);
  if (link_fused_ok(da)) {
    MTGNN_TRY(link_fused(z, n_q, max_q, da, p->W_d1, p->b_d1, p->W_d2, p->b_d2, L.Wp, L.DA, L.DB, L.part, dz, scores,
                         g->W_d2, g->b_d2, loss, s, prepared, s_dw != nullptr));
    // the partials' sums (loss, W_d2's gradient) and W_d1's gradient need only the fused kernel's outputs and
    // z: on the second stream if there is one
    if (s_dw) {
      hipError_t e = hipEventRecord(fork, s);
      if (e == hipSuccess) e = hipStreamWaitEvent(s_dw, fork, 0);
      if (e != hipSuccess) {
        set_hip_error(e, "link_loss fork");
        return MTGNN_EHIP;
      }
      MTGNN_TRY(link_reduce(L.part, n_q, max_q, da, g->W_d2, g->b_d2, loss, s_dw));
    }
    // DA is zero past the src block (the first third of the query rows), DB on it
    const DwProblem dp[2] = {{L.DA, da, z, da, g->W_d1, 2 * da, da, da, g->b_d1, 0, 1, 3},
                             {L.DB, da, z, da, g->W_d1 + da, 2 * da, da, da, L.db_scratch, 1, 3, 3}};
    return linear_dw_batch(dp, 2, max_q, n_q, MTGNN_F32, L.rest, L.rest_bytes, s_dw ? s_dw : s);
  }
  // general widths: the first layer's two halves over every query row
  const FwdProblem fp[2] = {{z, da, p->W_d1, 2 * da, nullptr, L.Y, 2 * da, da, da},
                            {z, da, p->W_d1 + da, 2 * da, nullptr, L.Y + da, 2 * da, da, da}};
  MTGNN_TRY(linear_fwd_batch(fp, 2, max_q, n_q, MTGNN_F32, MTGNN_F32, s));
  k_link_pairs<<<(unsigned)cdiv(max_tar < 1 ? 1 : max_tar, 4), 256, 0, s>>>(L.Y, n_q, max_tar, da, p->b_d1, p->W_d2,
                                                                              p->b_d2, L.DA, L.DB, L.Hp, L.n_tar,
                                                                              scores);
  MTGNN_CHECK_LAUNCH("link_pairs");
  MTGNN_TRY(colsum(L.Hp, da + 2, max_tar, L.n_tar, da + 2, L.sums, false, L.rest, L.rest_bytes, s));
  k_link_finish<<<1, 256, 0, s>>>(L.sums, da, g->W_d2, g->b_d2, loss);
  MTGNN_CHECK_LAUNCH("link_finish");
  // dW_d1 = [DA^T z | DB^T z], db_d1 = column sums of DA (the src rows carry dh_pos + dh_neg)
  const DwProblem dp[2] = {{L.DA, da, z, da, g->W_d1, 2 * da, da, da, g->b_d1},
                           {L.DB, da, z, da, g->W_d1 + da, 2 * da, da, da, L.db_scratch}};
  MTGNN_TRY(linear_dw_batch(dp, 2, max_q, n_q, MTGNN_F32, L.rest, L.rest_bytes, s));
  // dz = DA W_a + DB W_b over every query row
  MTGNN_TRY(linear_dx(L.DA, da, p->W_d1, MTGNN_F32, 2 * da, dz, da, max_q, n_q, da, da, false, s));
  MTGNN_TRY(linear_dx(L.DB, da, p->W_d1 + da, MTGNN_F32, 2 * da, dz, da, max_q, n_q, da, da, true, s));
  return MTGNN_OK;
}

}  // namespace mtgnn

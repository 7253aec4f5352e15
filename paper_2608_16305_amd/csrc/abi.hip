// C ABI of the mtgnn library: argument validation (host only, before any HIP
// call), workspace sizing, status strings, and dispatch to the step kernels.
#include <mutex>
#include <string>
#include <vector>

#include "ops.h"

namespace mtgnn {

static thread_local std::string g_err;

void set_hip_error(hipError_t e, const char* where) {
  g_err = std::string(where) + ": " + hipGetErrorString(e);
}

static mtgnn_status fail(mtgnn_status s, const char* what) {
  g_err = what;
  return s;
}

// ------------------------------------------------------------------ launch timer state

bool g_timer_armed = false;
static std::string g_timer_name;
static std::vector<hipEvent_t> g_timer_events;
static int g_timer_used = 0;

bool timer_begin(const char* name, hipStream_t s) {
  if (g_timer_used * 2 + 1 >= (int)g_timer_events.size() || g_timer_name != name) return false;
  return hipEventRecord(g_timer_events[2 * g_timer_used], s) == hipSuccess;
}

void timer_end(hipStream_t s) {
  (void)hipEventRecord(g_timer_events[2 * g_timer_used + 1], s);
  ++g_timer_used;
}

// Limits of this implementation (beyond them: MTGNN_EUNSUPPORTED).
constexpr int MAX_K = 64;          // one wave lane per neighbour slot
constexpr int MAX_HEAD_DIM = 128;  // two columns per lane
constexpr int MAX_SEG_WIDTH = 512; // d_mem + 2 d_attn, eight columns per lane

static mtgnn_status check_dims(const mtgnn_dims* d) {
  if (!d) return fail(MTGNN_EINVAL, "dims is NULL");
  if (d->dtype != MTGNN_F32 && d->dtype != MTGNN_BF16) return fail(MTGNN_EUNSUPPORTED, "dtype");
  if (d->n_nodes <= 0 || d->n_nodes >= (int64_t(1) << 31) - 1) return fail(MTGNN_EINVAL, "n_nodes");
  if (d->d_mem <= 0 || d->d_time < 0 || d->d_edge < 0 || d->d_attn <= 0 || d->n_heads <= 0 || d->k <= 0)
    return fail(MTGNN_EINVAL, "non-positive dimension");
  if (d->d_attn % d->n_heads != 0) return fail(MTGNN_EINVAL, "n_heads does not divide d_attn");
  if (d->k > MAX_K) return fail(MTGNN_EUNSUPPORTED, "k > 64");
  if (d->d_attn / d->n_heads > MAX_HEAD_DIM) return fail(MTGNN_EUNSUPPORTED, "head width > 128");
  if (d->d_mem + 2 * d->d_attn > MAX_SEG_WIDTH) return fail(MTGNN_EUNSUPPORTED, "d_mem + 2 d_attn > 512");
  return MTGNN_OK;
}

static mtgnn_status check_batch(const mtgnn_batch* b) {
  if (!b) return fail(MTGNN_EINVAL, "batch is NULL");
  if (b->n < 0 || b->n >= (int64_t(1) << 30)) return fail(MTGNN_EINVAL, "batch size");
  if (b->n > 0 && (!b->src || !b->dst || !b->t)) return fail(MTGNN_EINVAL, "batch src/dst/t NULL");
  return MTGNN_OK;
}

static mtgnn_status check_rows(int64_t max_rows) {
  if (max_rows < 0 || max_rows >= (int64_t(1) << 31) - 1) return fail(MTGNN_EINVAL, "max_rows");
  return MTGNN_OK;
}

#define REQ(p, name) \
  if (!(p)) return fail(MTGNN_EINVAL, name " is NULL")

// ------------------------------------------------------------------ allocation-free scratch

// Device-resident scratch of the allocation-free entry point.  Each GPU the library runs on holds its
// own copy for the life of the process.  In host code `scratch` names a host-side stand-in, never the
// device address: the address is taken once per device with hipGetSymbolAddress and only that pointer
// reaches kernels.
static __device__ __align__(256) unsigned char scratch[MTGNN_NOALLOC_SCRATCH_BYTES];

constexpr int MAX_DEVICES = 64;
static std::mutex g_scratch_mu;
static void* g_scratch_ptr[MAX_DEVICES] = {};

// The scratch address on the current device (looked up on the first call on that device).
static mtgnn_status scratch_on_current_device(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    set_hip_error(e, "hipGetDevice");
    return MTGNN_EHIP;
  }
  if (dev < 0 || dev >= MAX_DEVICES) return fail(MTGNN_EUNSUPPORTED, "device ordinal beyond 64");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      set_hip_error(e, "hipGetSymbolAddress(scratch)");
      return MTGNN_EHIP;
    }
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return MTGNN_OK;
}

}  // namespace mtgnn

using namespace mtgnn;

extern "C" {

int mtgnn_version(void) { return 100; }

const char* mtgnn_status_string(int status) {
  switch (status) {
    case MTGNN_OK: return "ok";
    case MTGNN_EINVAL: return "invalid argument";
    case MTGNN_EUNSUPPORTED: return "unsupported configuration";
    case MTGNN_EWORKSPACE: return "workspace too small";
    case MTGNN_EHIP: return "HIP error";
    default: return "unknown status";
  }
}

const char* mtgnn_last_error(void) { return g_err.c_str(); }

mtgnn_status mtgnn_timer_start(const char* kernel, int max_launches) {
  if (!kernel || max_launches <= 0 || max_launches > (1 << 20)) return fail(MTGNN_EINVAL, "timer arguments");
  if (g_timer_armed) return fail(MTGNN_EINVAL, "timer already running");
  g_timer_events.assign(2 * (size_t)max_launches, nullptr);
  for (auto& e : g_timer_events) {
    hipError_t err = hipEventCreate(&e);
    if (err != hipSuccess) {
      set_hip_error(err, "hipEventCreate");
      for (auto& x : g_timer_events)
        if (x) (void)hipEventDestroy(x);
      g_timer_events.clear();
      return MTGNN_EHIP;
    }
  }
  g_timer_name = kernel;
  g_timer_used = 0;
  g_timer_armed = true;
  return MTGNN_OK;
}

mtgnn_status mtgnn_timer_stop(double* total_ms, int* launches) {
  if (!g_timer_armed) return fail(MTGNN_EINVAL, "timer not running");
  g_timer_armed = false;
  double tot = 0.0;
  mtgnn_status st = MTGNN_OK;
  for (int i = 0; i < g_timer_used; ++i) {
    float ms = 0.f;
    hipError_t err = hipEventSynchronize(g_timer_events[2 * i + 1]);
    if (err == hipSuccess) err = hipEventElapsedTime(&ms, g_timer_events[2 * i], g_timer_events[2 * i + 1]);
    if (err != hipSuccess) {
      set_hip_error(err, "timer events");
      st = MTGNN_EHIP;
      break;
    }
    tot += ms;
  }
  for (auto& e : g_timer_events) (void)hipEventDestroy(e);
  g_timer_events.clear();
  if (total_ms) *total_ms = tot;
  if (launches) *launches = g_timer_used;
  g_timer_used = 0;
  return st;
}

size_t mtgnn_workspace_bytes(int op, const mtgnn_dims* d, int64_t max_rows, int64_t max_q) {
  if (max_rows < 0 || max_q < 0) return 0;
  switch (op) {
    case MTGNN_OP_BUILD_QUERIES: return build_queries_ws(max_rows);
    case MTGNN_OP_AGGREGATE_LAST: return aggregate_last_ws(max_rows, d ? d->n_nodes : 0);
    case MTGNN_OP_BUILD_MESSAGES: return 0;
    case MTGNN_OP_SAMPLE_RECENT: return 0;
    case MTGNN_OP_MIXED_BATCHES: return mixed_batches_ws(max_rows);
    case MTGNN_OP_BUILD_CSR: return build_csr_ws(max_rows, d ? d->n_nodes : 0);
    default: break;
  }
  if (check_dims(d) != MTGNN_OK) return 0;
  switch (op) {
    case MTGNN_OP_GRU_UPDATE: return gru_update_ws(d, max_rows);
    case MTGNN_OP_TEMPORAL_ATTN: return attn_fwd_ws(d, max_q);
    case MTGNN_OP_TEMPORAL_ATTN_BWD: return attn_bwd_ws(d, max_q, max_rows);
    case MTGNN_OP_GRU_UPDATE_BWD: return gru_update_bwd_ws(d, max_rows);
    case MTGNN_OP_BUILD_MESSAGES_BWD: return build_messages_bwd_ws(d, max_rows);
    case MTGNN_OP_LINK_LOSS: return link_loss_ws(d, max_q);
    case MTGNN_OP_RNN_UPDATE: return rnn_update_ws(d, max_rows);
    case MTGNN_OP_RNN_UPDATE_BWD: return rnn_update_bwd_ws(d, max_rows);
    case MTGNN_OP_TIME_PROJECTION_BWD: return time_projection_bwd_ws(d, max_q);
    default: return 0;
  }
}

size_t mtgnn_save_bytes(int op, const mtgnn_dims* d, int64_t max_rows, int64_t max_q) {
  if (check_dims(d) != MTGNN_OK || max_rows < 0 || max_q < 0) return 0;
  if (op == MTGNN_OP_GRU_UPDATE) return gru_save_bytes(d, max_rows);
  if (op == MTGNN_OP_RNN_UPDATE) return rnn_save_bytes(d, max_rows);
  if (op == MTGNN_OP_TEMPORAL_ATTN) return attn_save_bytes(d, max_q);
  return 0;
}

mtgnn_status mtgnn_build_queries(const mtgnn_batch* b, const int32_t* neg, int32_t* q_node, float* q_t, int32_t* n_q,
                                 void* ws, size_t ws_bytes, hipStream_t stream) {
  MTGNN_TRY(check_batch(b));
  REQ(neg || b->n == 0, "neg");
  REQ(q_node, "q_node");
  REQ(q_t, "q_t");
  REQ(n_q, "n_q");
  if (b->flags && b->n > 0 && ws_bytes < build_queries_ws(b->n)) return fail(MTGNN_EWORKSPACE, "build_queries ws");
  if (b->flags && b->n > 0 && !ws) return fail(MTGNN_EINVAL, "ws is NULL");
  return build_queries_impl(b, neg, q_node, q_t, n_q, ws, ws_bytes, stream);
}

mtgnn_status mtgnn_aggregate_last(const mtgnn_batch* b, int64_t n_nodes, int32_t* uniq, int32_t* winner,
                                  int32_t* n_uniq, void* ws, size_t ws_bytes, hipStream_t stream) {
  MTGNN_TRY(check_batch(b));
  if (n_nodes <= 0 || n_nodes >= (int64_t(1) << 31) - 1) return fail(MTGNN_EINVAL, "n_nodes");
  REQ(uniq, "uniq");
  REQ(winner, "winner");
  REQ(n_uniq, "n_uniq");
  if (ws_bytes < aggregate_last_ws(b->n, n_nodes)) return fail(MTGNN_EWORKSPACE, "aggregate_last ws");
  if (b->n > 0 && !ws) return fail(MTGNN_EINVAL, "ws is NULL");
  return aggregate_last_impl(b, n_nodes, uniq, winner, n_uniq, ws, ws_bytes, stream);
}

mtgnn_status mtgnn_build_messages(const mtgnn_batch* b, const int32_t* uniq, const int32_t* winner,
                                  const int32_t* n_rows, int64_t max_rows, const void* memory,
                                  const float* last_update, const float* edge_feat, const float* time_w,
                                  const float* time_b, const mtgnn_dims* d, void* msg, float* dt,
                                  hipStream_t stream) {
  MTGNN_TRY(check_batch(b));
  MTGNN_TRY(check_dims(d));
  MTGNN_TRY(check_rows(max_rows));
  REQ(uniq, "uniq");
  REQ(winner, "winner");
  REQ(memory, "memory");
  REQ(last_update, "last_update");
  REQ(msg, "msg");
  REQ(dt, "dt");
  if (d->d_time > 0 && (!time_w || !time_b)) return fail(MTGNN_EINVAL, "time encoder is NULL");
  if ((d->d_edge > 0) != (edge_feat != nullptr)) return fail(MTGNN_EINVAL, "edge_feat must be given iff d_edge > 0");
  if (d->d_edge > 0 && !b->eid && b->n > 0) return fail(MTGNN_EINVAL, "batch eid is NULL");
  if (max_rows == 0) return MTGNN_OK;
  return build_messages_impl(b, uniq, winner, n_rows, max_rows, memory, last_update, edge_feat, time_w, time_b, d, msg,
                             dt, stream);
}

mtgnn_status mtgnn_gru_update(const mtgnn_batch* b, const int32_t* uniq, const int32_t* winner,
                              const int32_t* n_rows, int64_t max_rows, const void* msg, const void* W_ih,
                              const void* W_hh, const float* b_ih, const float* b_hh, const mtgnn_dims* d,
                              void* memory, float* last_update, void* save, void* ws, size_t ws_bytes,
                              hipStream_t stream) {
  MTGNN_TRY(check_batch(b));
  MTGNN_TRY(check_dims(d));
  MTGNN_TRY(check_rows(max_rows));
  REQ(uniq, "uniq");
  REQ(winner, "winner");
  REQ(msg, "msg");
  REQ(W_ih, "W_ih");
  REQ(W_hh, "W_hh");
  REQ(b_ih, "b_ih");
  REQ(b_hh, "b_hh");
  REQ(memory, "memory");
  REQ(last_update, "last_update");
  if (ws_bytes < gru_update_ws(d, max_rows)) return fail(MTGNN_EWORKSPACE, "gru_update ws");
  if (max_rows == 0) return MTGNN_OK;
  REQ(ws, "ws");
  return gru_update_impl(b, uniq, winner, n_rows, max_rows, msg, W_ih, W_hh, b_ih, b_hh, d, memory, last_update, save,
                         ws, ws_bytes, stream);
}

mtgnn_status mtgnn_sample_recent(const int64_t* csr_off, const int32_t* csr_nbr, const float* csr_t,
                                 const int32_t* csr_eid, int64_t n_nodes, const int32_t* q_node, const float* q_t,
                                 const int32_t* n_q, int64_t max_q, int32_t k, int32_t* out_nbr, float* out_t,
                                 int32_t* out_eid, hipStream_t stream) {
  REQ(csr_off, "csr_off");
  REQ(csr_nbr, "csr_nbr");
  REQ(csr_t, "csr_t");
  REQ(csr_eid, "csr_eid");
  if (n_nodes <= 0) return fail(MTGNN_EINVAL, "n_nodes");
  if (max_q < 0 || max_q >= (int64_t(1) << 31) - 1) return fail(MTGNN_EINVAL, "max_q");
  if (k <= 0) return fail(MTGNN_EINVAL, "k");
  if (k > MAX_K) return fail(MTGNN_EUNSUPPORTED, "k > 64");
  if (max_q == 0) return MTGNN_OK;
  REQ(q_node, "q_node");
  REQ(q_t, "q_t");
  REQ(out_nbr, "out_nbr");
  REQ(out_t, "out_t");
  REQ(out_eid, "out_eid");
  return sample_recent_impl(csr_off, csr_nbr, csr_t, csr_eid, q_node, q_t, n_q, max_q, k, out_nbr, out_t, out_eid,
                            stream);
}

static mtgnn_status check_attn_params(const mtgnn_attn_params* p) {
  if (!p) return fail(MTGNN_EINVAL, "params is NULL");
  if (!p->W_q || !p->W_k || !p->W_v || !p->W_o || !p->W_1 || !p->W_2) return fail(MTGNN_EINVAL, "weight is NULL");
  if (!p->b_q || !p->b_k || !p->b_v || !p->b_o || !p->b_1 || !p->b_2) return fail(MTGNN_EINVAL, "bias is NULL");
  return MTGNN_OK;
}

static mtgnn_status attn_fwd_checked(const int32_t* q_node, const float* q_t, int64_t max_q, const int32_t* nbr,
                                     const float* nt, const int32_t* neid, const void* memory, const float* edge_feat,
                                     const float* time_w, const float* time_b, const mtgnn_attn_params* params,
                                     const mtgnn_dims* d, const float* z, const void* save) {
  MTGNN_TRY(check_dims(d));
  MTGNN_TRY(check_attn_params(params));
  if (max_q < 0 || max_q * (int64_t)d->k >= (int64_t(1) << 31) - 1) return fail(MTGNN_EINVAL, "max_q");
  if (max_q == 0) return MTGNN_OK;
  REQ(q_node, "q_node");
  REQ(q_t, "q_t");
  REQ(nbr, "nbr");
  REQ(nt, "nt");
  REQ(neid, "neid");
  REQ(memory, "memory");
  REQ(z, "z");
  REQ(save, "save");
  if (d->d_time > 0 && (!time_w || !time_b)) return fail(MTGNN_EINVAL, "time encoder is NULL");
  if ((d->d_edge > 0) != (edge_feat != nullptr)) return fail(MTGNN_EINVAL, "edge_feat must be given iff d_edge > 0");
  return MTGNN_OK;
}

mtgnn_status mtgnn_temporal_attn(const int32_t* q_node, const float* q_t, const int32_t* n_q, int64_t max_q,
                                 const int32_t* nbr, const float* nt, const int32_t* neid, const void* memory,
                                 const float* edge_feat, const float* time_w, const float* time_b,
                                 const mtgnn_attn_params* params, const mtgnn_dims* d, float* z, void* save, void* ws,
                                 size_t ws_bytes, hipStream_t stream) {
  MTGNN_TRY(attn_fwd_checked(q_node, q_t, max_q, nbr, nt, neid, memory, edge_feat, time_w, time_b, params, d, z,
                             save));
  if (max_q == 0) return MTGNN_OK;
  if (ws_bytes < attn_fwd_ws(d, max_q)) return fail(MTGNN_EWORKSPACE, "temporal_attn ws");
  return attn_fwd_impl(q_node, q_t, n_q, max_q, nbr, nt, neid, memory, edge_feat, time_w, time_b, params, d, z, save,
                       ws, ws_bytes, stream);
}

mtgnn_status mtgnn_temporal_attn_prepare(const int32_t* nbr, const int32_t* n_q, int64_t max_q,
                                         const mtgnn_attn_params* params, const float* time_w, const float* time_b,
                                         const mtgnn_dims* d, void* save, void* ws, size_t ws_bytes,
                                         hipStream_t stream) {
  MTGNN_TRY(check_dims(d));
  MTGNN_TRY(check_attn_params(params));
  if (max_q < 0 || max_q * (int64_t)d->k >= (int64_t(1) << 31) - 1) return fail(MTGNN_EINVAL, "max_q");
  if (max_q == 0) return MTGNN_OK;
  REQ(nbr, "nbr");
  REQ(save, "save");
  if (d->d_time > 0 && (!time_w || !time_b)) return fail(MTGNN_EINVAL, "time arrays");
  if (ws_bytes < attn_fwd_ws(d, max_q)) return fail(MTGNN_EWORKSPACE, "temporal_attn_prepare ws");
  return attn_prepare_impl(nbr, n_q, max_q, params, time_w, time_b, d, save, ws, ws_bytes, stream);
}

mtgnn_status mtgnn_temporal_attn_prepare_weights(const mtgnn_attn_params* params, const float* time_w,
                                                 const float* time_b, const mtgnn_dims* d, void* save,
                                                 hipStream_t stream) {
  MTGNN_TRY(check_dims(d));
  MTGNN_TRY(check_attn_params(params));
  REQ(save, "save");
  if (d->d_time > 0 && (!time_w || !time_b)) return fail(MTGNN_EINVAL, "time arrays");
  return attn_prepare_weights_impl(params, time_w, time_b, d, save, stream);
}

mtgnn_status mtgnn_temporal_attn_prepare_slots(const int32_t* nbr, const int32_t* n_q, int64_t max_q,
                                               const mtgnn_dims* d, void* save, void* ws, size_t ws_bytes,
                                               hipStream_t stream) {
  MTGNN_TRY(check_dims(d));
  if (max_q < 0 || max_q * (int64_t)d->k >= (int64_t(1) << 31) - 1) return fail(MTGNN_EINVAL, "max_q");
  if (max_q == 0) return MTGNN_OK;
  REQ(nbr, "nbr");
  REQ(save, "save");
  if (ws_bytes < attn_fwd_ws(d, max_q)) return fail(MTGNN_EWORKSPACE, "temporal_attn_prepare_slots ws");
  return attn_prepare_slots_impl(nbr, n_q, max_q, d, save, ws, ws_bytes, stream);
}

mtgnn_status mtgnn_temporal_attn_prepared(const int32_t* q_node, const float* q_t, const int32_t* n_q, int64_t max_q,
                                          const int32_t* nbr, const float* nt, const int32_t* neid,
                                          const void* memory, const float* edge_feat, const float* time_w,
                                          const float* time_b, const mtgnn_attn_params* params, const mtgnn_dims* d,
                                          float* z, void* save, hipStream_t stream) {
  MTGNN_TRY(attn_fwd_checked(q_node, q_t, max_q, nbr, nt, neid, memory, edge_feat, time_w, time_b, params, d, z,
                             save));
  if (max_q == 0) return MTGNN_OK;
  return attn_fwd_prepared_impl(q_node, q_t, n_q, max_q, nbr, nt, neid, memory, edge_feat, time_w, time_b, params, d,
                                z, save, stream);
}

static mtgnn_status attn_bwd_checked(const int32_t* q_node, const float* q_t, const int32_t* n_q, int64_t max_q,
                                     const int32_t* nbr, const float* nt, const float* dz, const void* save,
                                     const int32_t* uniq, const int32_t* n_rows, int64_t max_rows,
                                     const float* time_w, const float* time_b, const mtgnn_attn_params* params,
                                     const mtgnn_dims* d, mtgnn_attn_grads* g, float* d_mem, float* d_time_w,
                                     float* d_time_b, void* ws, size_t ws_bytes, hipStream_t stream,
                                     hipStream_t dmem_stream, hipEvent_t fork, hipEvent_t join,
                                     bool grouped = false) {
  MTGNN_TRY(check_dims(d));
  MTGNN_TRY(check_attn_params(params));
  MTGNN_TRY(check_rows(max_rows));
  if (max_q < 0 || max_q * (int64_t)d->k >= (int64_t(1) << 31) - 1) return fail(MTGNN_EINVAL, "max_q");
  if (!g || !g->W_q || !g->W_k || !g->W_v || !g->W_o || !g->W_1 || !g->W_2 || !g->b_q || !g->b_k || !g->b_v ||
      !g->b_o || !g->b_1 || !g->b_2)
    return fail(MTGNN_EINVAL, "grads");
  if (max_q == 0) return fail(MTGNN_EINVAL, "max_q == 0 (no query: every gradient is zero; skip the call)");
  REQ(q_node, "q_node");
  REQ(q_t, "q_t");
  REQ(nbr, "nbr");
  REQ(nt, "nt");
  REQ(dz, "dz");
  REQ(save, "save");
  if (max_rows > 0) {
    REQ(uniq, "uniq");
    REQ(d_mem, "d_mem");
  }
  if (d->d_time > 0 && (!time_w || !time_b || !d_time_w || !d_time_b)) return fail(MTGNN_EINVAL, "time arrays");
  if (ws_bytes < attn_bwd_ws(d, max_q, max_rows)) return fail(MTGNN_EWORKSPACE, "temporal_attn_bwd ws");
  REQ(ws, "ws");
  return attn_bwd_impl(q_node, q_t, n_q, max_q, nbr, nt, dz, save, uniq, n_rows, max_rows, time_w, time_b, params, d,
                       g, d_mem, d_time_w, d_time_b, ws, ws_bytes, stream, dmem_stream, fork, join, grouped);
}

mtgnn_status mtgnn_temporal_attn_bwd(const int32_t* q_node, const float* q_t, const int32_t* n_q, int64_t max_q,
                                     const int32_t* nbr, const float* nt, const float* dz, const void* save,
                                     const int32_t* uniq, const int32_t* n_rows, int64_t max_rows,
                                     const float* time_w, const float* time_b, const mtgnn_attn_params* params,
                                     const mtgnn_dims* d, mtgnn_attn_grads* g, float* d_mem, float* d_time_w,
                                     float* d_time_b, void* ws, size_t ws_bytes, hipStream_t stream) {
  return attn_bwd_checked(q_node, q_t, n_q, max_q, nbr, nt, dz, save, uniq, n_rows, max_rows, time_w, time_b, params,
                          d, g, d_mem, d_time_w, d_time_b, ws, ws_bytes, stream, nullptr, nullptr, nullptr);
}

mtgnn_status mtgnn_temporal_attn_bwd_overlap(const int32_t* q_node, const float* q_t, const int32_t* n_q,
                                             int64_t max_q, const int32_t* nbr, const float* nt, const float* dz,
                                             const void* save, const int32_t* uniq, const int32_t* n_rows,
                                             int64_t max_rows, const float* time_w, const float* time_b,
                                             const mtgnn_attn_params* params, const mtgnn_dims* d,
                                             mtgnn_attn_grads* g, float* d_mem, float* d_time_w, float* d_time_b,
                                             void* ws, size_t ws_bytes, hipStream_t stream, hipStream_t dmem_stream,
                                             hipEvent_t fork, hipEvent_t join) {
  if (max_rows > 0 && (!dmem_stream || !fork || !join))
    return fail(MTGNN_EINVAL, "temporal_attn_bwd_overlap: dmem_stream, fork and join are required");
  return attn_bwd_checked(q_node, q_t, n_q, max_q, nbr, nt, dz, save, uniq, n_rows, max_rows, time_w, time_b, params,
                          d, g, d_mem, d_time_w, d_time_b, ws, ws_bytes, stream, dmem_stream, fork, join);
}

mtgnn_status mtgnn_temporal_attn_bwd_group(const int32_t* q_node, const int32_t* n_q, int64_t max_q,
                                           const int32_t* nbr, const void* save, const int32_t* uniq,
                                           const int32_t* n_rows, int64_t max_rows, const mtgnn_dims* d, void* ws,
                                           size_t ws_bytes, hipStream_t stream) {
  MTGNN_TRY(check_dims(d));
  MTGNN_TRY(check_rows(max_rows));
  if (max_q <= 0 || max_q * (int64_t)d->k >= (int64_t(1) << 31) - 1) return fail(MTGNN_EINVAL, "max_q");
  REQ(q_node, "q_node");
  REQ(nbr, "nbr");
  REQ(save, "save");
  if (max_rows > 0) REQ(uniq, "uniq");
  if (ws_bytes < attn_bwd_ws(d, max_q, max_rows)) return fail(MTGNN_EWORKSPACE, "temporal_attn_bwd_group ws");
  REQ(ws, "ws");
  return attn_bwd_group_impl(q_node, n_q, max_q, nbr, save, uniq, n_rows, max_rows, d, ws, ws_bytes, stream);
}

mtgnn_status mtgnn_temporal_attn_bwd_grouped(const int32_t* q_node, const float* q_t, const int32_t* n_q,
                                             int64_t max_q, const int32_t* nbr, const float* nt, const float* dz,
                                             const void* save, const int32_t* uniq, const int32_t* n_rows,
                                             int64_t max_rows, const float* time_w, const float* time_b,
                                             const mtgnn_attn_params* params, const mtgnn_dims* d,
                                             mtgnn_attn_grads* g, float* d_mem, float* d_time_w, float* d_time_b,
                                             void* ws, size_t ws_bytes, hipStream_t stream, hipStream_t dmem_stream,
                                             hipEvent_t fork, hipEvent_t join) {
  if (max_rows > 0 && (!dmem_stream || !fork))
    return fail(MTGNN_EINVAL, "temporal_attn_bwd_grouped: dmem_stream and fork are required");
  return attn_bwd_checked(q_node, q_t, n_q, max_q, nbr, nt, dz, save, uniq, n_rows, max_rows, time_w, time_b, params,
                          d, g, d_mem, d_time_w, d_time_b, ws, ws_bytes, stream, dmem_stream, fork, join, true);
}

mtgnn_status mtgnn_gru_update_bwd(const float* d_mem, const void* save, const void* msg, const int32_t* n_rows,
                                  int64_t max_rows, const void* W_ih, const void* W_hh, const mtgnn_dims* d,
                                  float* dW_ih, float* dW_hh, float* db_ih, float* db_hh, float* dmsg_time, void* ws,
                                  size_t ws_bytes, hipStream_t stream) {
  MTGNN_TRY(check_dims(d));
  MTGNN_TRY(check_rows(max_rows));
  REQ(dW_ih, "dW_ih");
  REQ(dW_hh, "dW_hh");
  REQ(db_ih, "db_ih");
  REQ(db_hh, "db_hh");
  if (max_rows == 0) return fail(MTGNN_EINVAL, "max_rows == 0 (no updated row: every gradient is zero; skip the call)");
  REQ(d_mem, "d_mem");
  REQ(save, "save");
  REQ(msg, "msg");
  REQ(W_ih, "W_ih");
  REQ(W_hh, "W_hh");
  if (ws_bytes < gru_update_bwd_ws(d, max_rows)) return fail(MTGNN_EWORKSPACE, "gru_update_bwd ws");
  REQ(ws, "ws");
  return gru_update_bwd_impl(d_mem, save, msg, n_rows, max_rows, W_ih, W_hh, d, dW_ih, dW_hh, db_ih, db_hh, dmsg_time,
                             ws, ws_bytes, stream);
}

static mtgnn_status check_link_loss(const float* z, int64_t max_q, const mtgnn_link_params* params,
                                    const mtgnn_dims* d, float* loss, float* dz, mtgnn_link_grads* grads, void* ws,
                                    size_t ws_bytes) {
  MTGNN_TRY(check_dims(d));
  if (max_q < 0 || max_q >= (int64_t(1) << 31) - 1) return fail(MTGNN_EINVAL, "max_q");
  if (max_q % 3 != 0) return fail(MTGNN_EINVAL, "max_q is not a multiple of 3 (src, dst and negative blocks)");
  if (d->d_attn > 128) return fail(MTGNN_EUNSUPPORTED, "link_loss: d_attn > 128");
  REQ(params, "params");
  REQ(grads, "grads");
  REQ(params->W_d1, "W_d1");
  REQ(params->b_d1, "b_d1");
  REQ(params->W_d2, "W_d2");
  REQ(params->b_d2, "b_d2");
  REQ(grads->W_d1, "dW_d1");
  REQ(grads->b_d1, "db_d1");
  REQ(grads->W_d2, "dW_d2");
  REQ(grads->b_d2, "db_d2");
  REQ(loss, "loss");
  if (max_q > 0) {
    REQ(z, "z");
    REQ(dz, "dz");
  }
  if (ws_bytes < link_loss_ws(d, max_q)) return fail(MTGNN_EWORKSPACE, "link_loss ws");
  REQ(ws, "ws");
  return MTGNN_OK;
}

mtgnn_status mtgnn_link_loss(const float* z, const int32_t* n_q, int64_t max_q, const mtgnn_link_params* params,
                             const mtgnn_dims* d, float* loss, float* scores, float* dz, mtgnn_link_grads* grads,
                             void* ws, size_t ws_bytes, hipStream_t stream) {
  MTGNN_TRY(check_link_loss(z, max_q, params, d, loss, dz, grads, ws, ws_bytes));
  return link_loss_impl(z, n_q, max_q, params, d, loss, scores, dz, grads, ws, ws_bytes, stream);
}

mtgnn_status mtgnn_link_loss_overlap(const float* z, const int32_t* n_q, int64_t max_q,
                                     const mtgnn_link_params* params, const mtgnn_dims* d, float* loss, float* scores,
                                     float* dz, mtgnn_link_grads* grads, void* ws, size_t ws_bytes,
                                     hipStream_t stream, hipStream_t dw_stream, hipEvent_t fork) {
  MTGNN_TRY(check_link_loss(z, max_q, params, d, loss, dz, grads, ws, ws_bytes));
  REQ(dw_stream, "dw_stream");
  REQ(fork, "fork");
  return link_loss_impl(z, n_q, max_q, params, d, loss, scores, dz, grads, ws, ws_bytes, stream, dw_stream, fork);
}

mtgnn_status mtgnn_link_prepare_weights(const mtgnn_link_params* params, const mtgnn_dims* d, int64_t max_q, void* ws,
                                        size_t ws_bytes, hipStream_t stream) {
  MTGNN_TRY(check_dims(d));
  if (max_q < 0 || max_q >= (int64_t(1) << 31) - 1) return fail(MTGNN_EINVAL, "max_q");
  if (max_q % 3 != 0) return fail(MTGNN_EINVAL, "max_q is not a multiple of 3 (src, dst and negative blocks)");
  if (d->d_attn > 128) return fail(MTGNN_EUNSUPPORTED, "link_prepare_weights: d_attn > 128");
  REQ(params, "params");
  REQ(params->W_d1, "W_d1");
  if (ws_bytes < link_loss_ws(d, max_q)) return fail(MTGNN_EWORKSPACE, "link_prepare_weights ws");
  REQ(ws, "ws");
  return link_prepare_impl(params, d, max_q, ws, stream);
}

mtgnn_status mtgnn_temporal_attn_prepare_weights_link(const mtgnn_attn_params* params, const float* time_w,
                                                      const float* time_b, const mtgnn_dims* d, void* save,
                                                      const mtgnn_link_params* link, int64_t max_q, void* link_ws,
                                                      size_t link_ws_bytes, hipStream_t stream) {
  MTGNN_TRY(check_dims(d));
  MTGNN_TRY(check_attn_params(params));
  REQ(save, "save");
  if (d->d_time > 0 && (!time_w || !time_b)) return fail(MTGNN_EINVAL, "time arrays");
  if (max_q < 0 || max_q >= (int64_t(1) << 31) - 1) return fail(MTGNN_EINVAL, "max_q");
  if (max_q % 3 != 0) return fail(MTGNN_EINVAL, "max_q is not a multiple of 3 (src, dst and negative blocks)");
  if (d->d_attn > 128) return fail(MTGNN_EUNSUPPORTED, "link weights: d_attn > 128");
  REQ(link, "link");
  REQ(link->W_d1, "W_d1");
  if (link_ws_bytes < link_loss_ws(d, max_q)) return fail(MTGNN_EWORKSPACE, "link ws");
  REQ(link_ws, "link_ws");
  PadCopy c[4];
  const int n = link_copies_impl(link, d, max_q, link_ws, c);
  return attn_prepare_weights_impl(params, time_w, time_b, d, save, stream, c, n);
}

mtgnn_status mtgnn_link_loss_prepared(const float* z, const int32_t* n_q, int64_t max_q,
                                      const mtgnn_link_params* params, const mtgnn_dims* d, float* loss,
                                      float* scores, float* dz, mtgnn_link_grads* grads, void* ws, size_t ws_bytes,
                                      hipStream_t stream, hipStream_t dw_stream, hipEvent_t fork) {
  MTGNN_TRY(check_link_loss(z, max_q, params, d, loss, dz, grads, ws, ws_bytes));
  if ((dw_stream == nullptr) != (fork == nullptr)) return fail(MTGNN_EINVAL, "dw_stream and fork: both or neither");
  return link_loss_impl(z, n_q, max_q, params, d, loss, scores, dz, grads, ws, ws_bytes, stream, dw_stream, fork,
                        true);
}

mtgnn_status mtgnn_build_messages_bwd(const float* dmsg_time, const float* dt, const int32_t* n_rows,
                                      int64_t max_rows, const float* time_w, const float* time_b, const mtgnn_dims* d,
                                      float* d_time_w, float* d_time_b, void* ws, size_t ws_bytes,
                                      hipStream_t stream) {
  MTGNN_TRY(check_dims(d));
  MTGNN_TRY(check_rows(max_rows));
  if (max_rows == 0 || d->d_time == 0) return MTGNN_OK;
  REQ(dmsg_time, "dmsg_time");
  REQ(dt, "dt");
  REQ(time_w, "time_w");
  REQ(time_b, "time_b");
  REQ(d_time_w, "d_time_w");
  REQ(d_time_b, "d_time_b");
  if (ws_bytes < build_messages_bwd_ws(d, max_rows)) return fail(MTGNN_EWORKSPACE, "build_messages_bwd ws");
  REQ(ws, "ws");
  return build_messages_bwd_impl(dmsg_time, dt, n_rows, max_rows, time_w, time_b, d, d_time_w, d_time_b, ws, ws_bytes,
                                 stream);
}

mtgnn_status mtgnn_build_messages_bwd_noalloc(const float* dmsg_time, const float* dt, const int32_t* n_rows,
                                              int64_t max_rows, const float* time_w, const float* time_b,
                                              const mtgnn_dims* d, float* d_time_w, float* d_time_b,
                                              hipStream_t stream) {
  MTGNN_TRY(check_dims(d));
  MTGNN_TRY(check_rows(max_rows));
  if (max_rows == 0 || d->d_time == 0) return MTGNN_OK;
  REQ(dmsg_time, "dmsg_time");
  REQ(dt, "dt");
  REQ(time_w, "time_w");
  REQ(time_b, "time_b");
  REQ(d_time_w, "d_time_w");
  REQ(d_time_b, "d_time_b");
  const size_t need = build_messages_bwd_ws(d, max_rows);
  if (need > (size_t)MTGNN_NOALLOC_SCRATCH_BYTES)
    return fail(MTGNN_EWORKSPACE, "build_messages_bwd_noalloc: 8 * d_time * ceil(max_rows / 32) bytes exceed the "
                                  "4 MiB device scratch");
  if (stream) {
    int cur = -1, sdev = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e == hipSuccess) e = hipStreamGetDevice(stream, &sdev);
    if (e != hipSuccess) {
      set_hip_error(e, "stream device");
      return MTGNN_EHIP;
    }
    if (sdev != cur) return fail(MTGNN_EINVAL, "stream is not on the current device");
  }
  void* ws = nullptr;
  MTGNN_TRY(scratch_on_current_device(&ws));
  return build_messages_bwd_impl(dmsg_time, dt, n_rows, max_rows, time_w, time_b, d, d_time_w, d_time_b, ws,
                                 (size_t)MTGNN_NOALLOC_SCRATCH_BYTES, stream);
}

mtgnn_status mtgnn_dependency_scan(const int32_t* src, const int32_t* dst, int64_t n_events, const int32_t* owner,
                                   int64_t n_nodes, int32_t n_workers, int64_t batch, int32_t window, uint8_t* role,
                                   uint32_t* sync_bits, hipStream_t stream) {
  if (n_events < 0 || n_events >= (int64_t(1) << 31) - 1) return fail(MTGNN_EINVAL, "n_events");
  if (n_nodes <= 0 || n_nodes >= (int64_t(1) << 31) - 1) return fail(MTGNN_EINVAL, "n_nodes");
  if (n_workers <= 0 || n_workers > 4096) return fail(MTGNN_EINVAL, "n_workers");
  if (batch <= 0 || window <= 0) return fail(MTGNN_EINVAL, "batch / window");
  if (n_events == 0) return MTGNN_OK;
  if ((int64_t)n_workers * cdiv(cdiv(n_events, batch), window) >= (int64_t(1) << 31))
    return fail(MTGNN_EINVAL, "too many (worker, window) scans");
  REQ(src, "src");
  REQ(dst, "dst");
  REQ(owner, "owner");
  REQ(role, "role");
  REQ(sync_bits, "sync_bits");
  return dep_scan_impl(src, dst, n_events, owner, n_nodes, n_workers, batch, window, role, sync_bits, stream);
}

mtgnn_status mtgnn_mixed_batches(const uint8_t* role, int64_t n_events, int64_t batch, int32_t* eid_out,
                                 uint8_t* flags_out, int32_t* batch_off, void* ws, size_t ws_bytes,
                                 hipStream_t stream) {
  if (n_events < 0 || n_events >= (int64_t(1) << 31) - 1) return fail(MTGNN_EINVAL, "n_events");
  if (batch <= 0) return fail(MTGNN_EINVAL, "batch");
  REQ(batch_off, "batch_off");
  if (n_events > 0) {
    REQ(role, "role");
    REQ(eid_out, "eid_out");
    REQ(flags_out, "flags_out");
    REQ(ws, "ws");
  }
  if (ws_bytes < mixed_batches_ws(n_events)) return fail(MTGNN_EWORKSPACE, "mixed_batches ws");
  return mixed_batches_impl(role, n_events, batch, eid_out, flags_out, batch_off, ws, ws_bytes, stream);
}

static mtgnn_status check_tensor_list(const void* const* ptrs, const int64_t* sizes, int32_t n) {
  if (!ptrs || !sizes) return fail(MTGNN_EINVAL, "tensor list is NULL");
  if (n <= 0 || n > RT_MAX_TENSORS) return fail(MTGNN_EINVAL, "tensor count not in 1..32");
  for (int i = 0; i < n; ++i) {
    if (!ptrs[i]) return fail(MTGNN_EINVAL, "tensor pointer is NULL");
    if (sizes[i] <= 0 || sizes[i] >= (int64_t(1) << 40)) return fail(MTGNN_EINVAL, "tensor size");
  }
  return MTGNN_OK;
}

size_t mtgnn_grad_norm_ws_bytes(const int64_t* sizes, int32_t n) {
  if (!sizes || n <= 0 || n > RT_MAX_TENSORS) return 0;
  return grad_norm_ws(sizes, n);
}

mtgnn_status mtgnn_grad_norm(const float* const* grads, const int64_t* sizes, int32_t n, double* norm, void* ws,
                             size_t ws_bytes, hipStream_t stream) {
  MTGNN_TRY(check_tensor_list((const void* const*)grads, sizes, n));
  REQ(norm, "norm");
  REQ(ws, "ws");
  if (ws_bytes < grad_norm_ws(sizes, n)) return fail(MTGNN_EWORKSPACE, "grad_norm ws");
  return grad_norm_impl(grads, sizes, n, norm, ws, stream);
}

mtgnn_status mtgnn_prune_aux(uint8_t* flags, int64_t n, int32_t heavy, hipStream_t stream) {
  if (n < 0) return fail(MTGNN_EINVAL, "n");
  if (n > 0) REQ(flags, "flags");
  return prune_aux_impl(flags, n, heavy, stream);
}

mtgnn_status mtgnn_cache_refresh(const uint32_t* sync_bits, int64_t n_nodes, const void* auth_memory,
                                 const float* auth_last_update, const mtgnn_dims* d, void* memory,
                                 float* last_update, hipStream_t stream) {
  MTGNN_TRY(check_dims(d));
  if (n_nodes <= 0 || n_nodes > d->n_nodes) return fail(MTGNN_EINVAL, "n_nodes");
  REQ(sync_bits, "sync_bits");
  REQ(auth_memory, "auth_memory");
  REQ(auth_last_update, "auth_last_update");
  REQ(memory, "memory");
  REQ(last_update, "last_update");
  return cache_refresh_impl(sync_bits, n_nodes, auth_memory, auth_last_update, d, memory, last_update, stream);
}

mtgnn_status mtgnn_adam_step(float* const* params, const float* const* grads, float* const* m, float* const* v,
                             void* const* shadow, const int64_t* sizes, int32_t n, const mtgnn_adam_config* cfg,
                             hipStream_t stream) {
  MTGNN_TRY(check_tensor_list((const void* const*)params, sizes, n));
  MTGNN_TRY(check_tensor_list((const void* const*)grads, sizes, n));
  MTGNN_TRY(check_tensor_list((const void* const*)m, sizes, n));
  MTGNN_TRY(check_tensor_list((const void* const*)v, sizes, n));
  REQ(cfg, "cfg");
  if (cfg->t < 1 || !(cfg->lr >= 0) || !(cfg->beta1 >= 0 && cfg->beta1 < 1) || !(cfg->beta2 >= 0 && cfg->beta2 < 1) ||
      !(cfg->eps > 0))
    return fail(MTGNN_EINVAL, "adam config");
  return adam_impl(params, grads, m, v, shadow, sizes, n, cfg, stream);
}

mtgnn_status mtgnn_rnn_update(const mtgnn_batch* b, const int32_t* uniq, const int32_t* winner,
                              const int32_t* n_rows, int64_t max_rows, const void* msg, const void* W_ih,
                              const void* W_hh, const float* b_ih, const float* b_hh, const mtgnn_dims* d,
                              void* memory, float* last_update, void* save, void* ws, size_t ws_bytes,
                              hipStream_t stream) {
  MTGNN_TRY(check_dims(d));
  MTGNN_TRY(check_batch(b));
  MTGNN_TRY(check_rows(max_rows));
  if (d->d_mem > 256) return fail(MTGNN_EUNSUPPORTED, "rnn_update: d_mem > 256");
  if (max_rows == 0) return MTGNN_OK;
  REQ(uniq, "uniq");
  REQ(winner, "winner");
  REQ(msg, "msg");
  REQ(W_ih, "W_ih");
  REQ(W_hh, "W_hh");
  REQ(b_ih, "b_ih");
  REQ(b_hh, "b_hh");
  REQ(memory, "memory");
  REQ(last_update, "last_update");
  if (ws_bytes < rnn_update_ws(d, max_rows)) return fail(MTGNN_EWORKSPACE, "rnn_update ws");
  REQ(ws, "ws");
  return rnn_update_impl(b, uniq, winner, n_rows, max_rows, msg, W_ih, W_hh, b_ih, b_hh, d, memory, last_update, save,
                         ws, ws_bytes, stream);
}

mtgnn_status mtgnn_rnn_update_bwd(const float* d_mem, const void* save, const void* msg, const int32_t* n_rows,
                                  int64_t max_rows, const void* W_ih, const void* W_hh, const mtgnn_dims* d,
                                  float* dW_ih, float* dW_hh, float* db_ih, float* db_hh, float* dmsg_time,
                                  void* ws, size_t ws_bytes, hipStream_t stream) {
  MTGNN_TRY(check_dims(d));
  MTGNN_TRY(check_rows(max_rows));
  REQ(dW_ih, "dW_ih");
  REQ(dW_hh, "dW_hh");
  REQ(db_ih, "db_ih");
  REQ(db_hh, "db_hh");
  if (max_rows == 0) return fail(MTGNN_EINVAL, "max_rows == 0 (no updated row: every gradient is zero; skip the call)");
  REQ(d_mem, "d_mem");
  REQ(save, "save");
  REQ(msg, "msg");
  REQ(W_ih, "W_ih");
  if (ws_bytes < rnn_update_bwd_ws(d, max_rows)) return fail(MTGNN_EWORKSPACE, "rnn_update_bwd ws");
  REQ(ws, "ws");
  return rnn_update_bwd_impl(d_mem, save, msg, n_rows, max_rows, W_ih, W_hh, d, dW_ih, dW_hh, db_ih, db_hh, dmsg_time,
                             ws, ws_bytes, stream);
}

mtgnn_status mtgnn_time_projection(const int32_t* q_node, const float* q_t, const int32_t* n_q, int64_t max_q,
                                   const void* memory, const float* last_update, const float* W_p, const float* b_p,
                                   float time_scale, const mtgnn_dims* d, float* z, hipStream_t stream) {
  MTGNN_TRY(check_dims(d));
  if (max_q < 0 || max_q >= (int64_t(1) << 31) - 1) return fail(MTGNN_EINVAL, "max_q");
  if (max_q == 0) return MTGNN_OK;
  REQ(q_node, "q_node");
  REQ(q_t, "q_t");
  REQ(memory, "memory");
  REQ(last_update, "last_update");
  REQ(W_p, "W_p");
  REQ(b_p, "b_p");
  REQ(z, "z");
  return time_projection_impl(q_node, q_t, n_q, max_q, memory, last_update, W_p, b_p, time_scale, d, z, stream);
}

mtgnn_status mtgnn_time_projection_bwd(const int32_t* q_node, const float* q_t, const int32_t* n_q, int64_t max_q,
                                       const void* memory, const float* last_update, const float* W_p,
                                       const float* b_p, float time_scale, const float* dz, const int32_t* uniq,
                                       const int32_t* n_rows, int64_t max_rows, const mtgnn_dims* d, float* dW_p,
                                       float* db_p, float* d_mem, void* ws, size_t ws_bytes, hipStream_t stream) {
  MTGNN_TRY(check_dims(d));
  MTGNN_TRY(check_rows(max_rows));
  if (d->d_mem > 256) return fail(MTGNN_EUNSUPPORTED, "time_projection_bwd: d_mem > 256");
  if (max_q < 0 || max_q >= (int64_t(1) << 31) - 1) return fail(MTGNN_EINVAL, "max_q");
  REQ(dW_p, "dW_p");
  REQ(db_p, "db_p");
  REQ(W_p, "W_p");
  REQ(b_p, "b_p");
  if (max_q > 0) {
    REQ(q_node, "q_node");
    REQ(q_t, "q_t");
    REQ(memory, "memory");
    REQ(last_update, "last_update");
    REQ(dz, "dz");
  }
  if (max_rows > 0) {
    REQ(uniq, "uniq");
    REQ(d_mem, "d_mem");
  }
  if (ws_bytes < time_projection_bwd_ws(d, max_q)) return fail(MTGNN_EWORKSPACE, "time_projection_bwd ws");
  REQ(ws, "ws");
  return time_projection_bwd_impl(q_node, q_t, n_q, max_q, memory, last_update, W_p, b_p, time_scale, dz, uniq, n_rows,
                                  max_rows, d, dW_p, db_p, d_mem, ws, ws_bytes, stream);
}

mtgnn_status mtgnn_build_temporal_csr(const int32_t* src, const int32_t* dst, const float* t, int64_t n_events,
                                      int64_t n_nodes, int64_t* csr_off, int32_t* csr_nbr, float* csr_t,
                                      int32_t* csr_eid, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (n_events < 0 || n_events >= (int64_t(1) << 31) - 1) return fail(MTGNN_EINVAL, "n_events");
  if (n_nodes <= 0 || n_nodes >= (int64_t(1) << 31) - 1) return fail(MTGNN_EINVAL, "n_nodes");
  REQ(csr_off, "csr_off");
  if (n_events > 0) {
    REQ(src, "src");
    REQ(dst, "dst");
    REQ(t, "t");
    REQ(csr_nbr, "csr_nbr");
    REQ(csr_t, "csr_t");
    REQ(csr_eid, "csr_eid");
    REQ(ws, "ws");
  }
  if (ws_bytes < build_csr_ws(n_events, n_nodes)) return fail(MTGNN_EWORKSPACE, "build_csr ws");
  return build_csr_impl(src, dst, t, n_events, n_nodes, csr_off, csr_nbr, csr_t, csr_eid, ws, ws_bytes, stream);
}

}  // extern "C"

// Internal entry points behind the C ABI (validation happens in abi.cpp).
#pragma once

#include "common.h"

namespace mtgnn {

// batch intake / memory phase
size_t build_queries_ws(int64_t n);
mtgnn_status build_queries_impl(const mtgnn_batch* b, const int32_t* neg, int32_t* q_node, float* q_t, int32_t* n_q,
                                void* ws, size_t ws_bytes, hipStream_t s);
size_t aggregate_last_ws(int64_t n, int64_t n_nodes);
mtgnn_status aggregate_last_impl(const mtgnn_batch* b, int64_t n_nodes, int32_t* uniq, int32_t* winner,
                                 int32_t* n_uniq, void* ws, size_t ws_bytes, hipStream_t s);
mtgnn_status build_messages_impl(const mtgnn_batch* b, const int32_t* uniq, const int32_t* winner,
                                 const int32_t* n_rows, int64_t max_rows, const void* memory, const float* lu,
                                 const float* edge_feat, const float* tw, const float* tb, const mtgnn_dims* d,
                                 void* msg, float* dt, hipStream_t s);
size_t gru_save_bytes(const mtgnn_dims* d, int64_t max_rows);
size_t gru_update_ws(const mtgnn_dims* d, int64_t max_rows);
mtgnn_status gru_update_impl(const mtgnn_batch* b, const int32_t* uniq, const int32_t* winner, const int32_t* n_rows,
                             int64_t max_rows, const void* msg, const void* W_ih, const void* W_hh, const float* b_ih,
                             const float* b_hh, const mtgnn_dims* d, void* memory, float* lu, void* save, void* ws,
                             size_t ws_bytes, hipStream_t s);
size_t gru_update_bwd_ws(const mtgnn_dims* d, int64_t max_rows);
mtgnn_status gru_update_bwd_impl(const float* d_mem, const void* save, const void* msg, const int32_t* n_rows,
                                 int64_t max_rows, const void* W_ih, const void* W_hh, const mtgnn_dims* d,
                                 float* dW_ih, float* dW_hh, float* db_ih, float* db_hh, float* dmsg_time, void* ws,
                                 size_t ws_bytes, hipStream_t s);
size_t build_messages_bwd_ws(const mtgnn_dims* d, int64_t max_rows);
mtgnn_status build_messages_bwd_impl(const float* dmsg_time, const float* dt, const int32_t* n_rows, int64_t max_rows,
                                     const float* tw, const float* tb, const mtgnn_dims* d, float* dw, float* db,
                                     void* ws, size_t ws_bytes, hipStream_t s);

// time-encoder gradient reductions (fixed order)
size_t timegrad_ws_bytes(int64_t rows, int dt_dim);
// d_time_w[j] (+)= sum_r dphi[r,j] (-sin(arg_rj)) delta_r,  d_time_b[j] (+)= sum_r dphi[r,j] (-sin(arg_rj)),
// arg_rj = time_w[j] delta_r + time_b[j]; delta == nullptr means delta_r = 0; sin_saved (optional) holds
// sin(arg) per [row, j]; rows are clamped by rows_dev.
// Sums the per-block partials [blocks][2][dt_dim] of a time-gradient GEMM epilogue
// (blocks = ceil(rows / chunk_rows), rows clamped by rows_dev) into dw, db.
mtgnn_status timegrad_reduce_blocks(const float* part, int64_t rows, const int32_t* rows_dev, int chunk_rows,
                                    int dt_dim, float* dw, float* db, bool accumulate, hipStream_t s);
// dw = (sum over p1's row chunks) + (sum over p2's), in one launch (the same bits as two reduces,
// the first overwriting, the second accumulating).
mtgnn_status timegrad_reduce_blocks2(const float* p1, int64_t rows1, const int32_t* rows_dev1, const float* p2,
                                     int64_t rows2, const int32_t* rows_dev2, int chunk_rows, int dt_dim, float* dw,
                                     float* db, hipStream_t s);
// dw = the slots' sum; db = the slots' sum + the queries' closed-form share (their time input is
// phi(0)): -sin(b_j) sum_a dbq[a] Wq[a * ldw + col0 + j] (float32 weights); and the query weight's
// time columns dWq[a * ldw + col0 + j] = dbq[a] phi(0)_j.
mtgnn_status timegrad_reduce_slots_q(const float* part, int64_t rows, const int32_t* rows_dev, int chunk_rows,
                                     int dt_dim, const float* dbq, const float* Wq, int64_t ldw, int col0, int da,
                                     const float* tw, const float* tb, float* dw, float* db, float* dWq,
                                     hipStream_t s);
mtgnn_status timegrad_rows(const float* dphi, int64_t ld, int64_t rows, const int32_t* rows_dev, const float* delta,
                           const float* sin_saved, const float* tw, const float* tb, int dt_dim, float* dw, float* db,
                           bool accumulate, void* ws, size_t ws_bytes, hipStream_t s);

// The GRU update fused on the layer machinery (merge.hip), float32: both products and the gates per block
// of 16 rows x 32 hidden units, from zero-padded per-group weight copies (Wp: gru_fused_weight_floats) that
// the same call writes first; wt (optional) is the backward's padded W_ih time slice, written alongside.
struct GruWTArgs {
  float* dst;
  int rows, cols, dt, K, ld, col0;
};
bool gru_fused_ok(int dtype, int dm, int dmsg);
size_t gru_fused_weight_floats(int dm, int dmsg);
mtgnn_status gru_fused(const float* msg, const float* W_ih, const float* W_hh, const float* b_ih, const float* b_hh,
                       const int32_t* uniq, const int32_t* winner, const float* t, const int32_t* n_rows,
                       int64_t max_rows, int dm, int dmsg, float* Wp, float* mem, float* lu, float* sr, float* sz,
                       float* sn, float* sghn, GruWTArgs wt, hipStream_t s);

// link-prediction decoder and the masked batch loss
// The fused form (merge.hip) for d_attn = 100 or 32: one kernel per 16 target events for the forward, the
// loss terms and dz, and the hidden-row gradients DA / DB for the first layer's weight gradient; then the
// column sums of the per-block partials into dW_d2, db_d2 and the loss.  Wp: link_fused_weight_floats.
bool link_fused_ok(int da);
size_t link_fused_weight_floats(int da);
// prepared: Wp already holds link_prepare_weights' copies of this W1 (else they are made first).
// s_reduce: the caller launches link_reduce itself (on another stream ordered after this call's work).
mtgnn_status link_fused(const float* z, const int32_t* n_q, int64_t max_q, int da, const float* W1, const float* b1,
                        const float* W2, const float* b2, float* Wp, float* DA, float* DB, float* part, float* dz,
                        float* scores, float* dW2, float* db2, float* loss, hipStream_t s, bool prepared = false,
                        bool s_reduce = false);
// The fixed-order sums of link_fused's per-block partials into dW_d2, db_d2 and the loss.
mtgnn_status link_reduce(const float* part, const int32_t* n_q, int64_t max_q, int da, float* dW2, float* db2,
                         float* loss, hipStream_t s);

size_t link_loss_ws(const mtgnn_dims* d, int64_t max_q);
// s_dw, fork: a second stream and an event (or NULL, NULL): W_d1's gradient is then enqueued on s_dw after
// fork, recorded on s once dz and the decoder's row gradients are written (fused widths only).
// prepared: link_prepare_impl has filled ws's weight copies from p (same max_q), ordered before this call.
mtgnn_status link_loss_impl(const float* z, const int32_t* n_q, int64_t max_q, const mtgnn_link_params* p,
                            const mtgnn_dims* d, float* loss, float* scores, float* dz, mtgnn_link_grads* g, void* ws,
                            size_t ws_bytes, hipStream_t s, hipStream_t s_dw = nullptr, hipEvent_t fork = nullptr,
                            bool prepared = false);


// offline dependency scan (Algorithm 1) and the mixed batches of one worker
mtgnn_status dep_scan_impl(const int32_t* src, const int32_t* dst, int64_t E, const int32_t* owner, int64_t n_nodes,
                           int n_workers, int64_t batch, int window, uint8_t* role, uint32_t* sync, hipStream_t s);
size_t mixed_batches_ws(int64_t E);
mtgnn_status mixed_batches_impl(const uint8_t* role, int64_t E, int64_t batch, int32_t* eid_out, uint8_t* flags_out,
                                int32_t* batch_off, void* ws, size_t ws_bytes, hipStream_t s);

// runtime controller's device work (runtime.hip)
constexpr int RT_MAX_TENSORS = 32;
size_t grad_norm_ws(const int64_t* sizes, int n);
mtgnn_status grad_norm_impl(const float* const* grads, const int64_t* sizes, int n, double* norm, void* ws,
                            hipStream_t s);
mtgnn_status prune_aux_impl(uint8_t* flags, int64_t n, int heavy, hipStream_t s);
mtgnn_status cache_refresh_impl(const uint32_t* bits, int64_t n_nodes, const void* auth_mem, const float* auth_lu,
                                const mtgnn_dims* d, void* mem, float* lu, hipStream_t s);
mtgnn_status adam_impl(float* const* params, const float* const* grads, float* const* m, float* const* v,
                       void* const* shadow, const int64_t* sizes, int n, const mtgnn_adam_config* c, hipStream_t s);

// the JODIE variant (jodie.hip)
size_t rnn_save_bytes(const mtgnn_dims* d, int64_t max_rows);
size_t rnn_update_ws(const mtgnn_dims* d, int64_t max_rows);
mtgnn_status rnn_update_impl(const mtgnn_batch* b, const int32_t* uniq, const int32_t* winner, const int32_t* n_rows,
                             int64_t max_rows, const void* msg, const void* W_ih, const void* W_hh, const float* b_ih,
                             const float* b_hh, const mtgnn_dims* d, void* memory, float* lu, void* save, void* ws,
                             size_t ws_bytes, hipStream_t s);
size_t rnn_update_bwd_ws(const mtgnn_dims* d, int64_t max_rows);
mtgnn_status rnn_update_bwd_impl(const float* d_mem, const void* save, const void* msg, const int32_t* n_rows,
                                 int64_t max_rows, const void* W_ih, const void* W_hh, const mtgnn_dims* d,
                                 float* dW_ih, float* dW_hh, float* db_ih, float* db_hh, float* dmsg_time, void* ws,
                                 size_t ws_bytes, hipStream_t s);
mtgnn_status time_projection_impl(const int32_t* q_node, const float* q_t, const int32_t* n_q, int64_t max_q,
                                  const void* memory, const float* lu, const float* Wp, const float* bp, float scale,
                                  const mtgnn_dims* d, float* z, hipStream_t s);
size_t time_projection_bwd_ws(const mtgnn_dims* d, int64_t max_q);
mtgnn_status time_projection_bwd_impl(const int32_t* q_node, const float* q_t, const int32_t* n_q, int64_t max_q,
                                      const void* memory, const float* lu, const float* Wp, const float* bp,
                                      float scale, const float* dz, const int32_t* uniq, const int32_t* n_rows,
                                      int64_t max_rows, const mtgnn_dims* d, float* dWp, float* dbp, float* d_mem,
                                      void* ws, size_t ws_bytes, hipStream_t s);

// sampling / adjacency
mtgnn_status sample_recent_impl(const int64_t* off, const int32_t* nbr, const float* t, const int32_t* eid,
                                const int32_t* q_node, const float* q_t, const int32_t* n_q, int64_t max_q, int k,
                                int32_t* out_nbr, float* out_t, int32_t* out_eid, hipStream_t s);
size_t build_csr_ws(int64_t n_events, int64_t n_nodes);
mtgnn_status build_csr_impl(const int32_t* src, const int32_t* dst, const float* t, int64_t n_events, int64_t n_nodes,
                            int64_t* off, int32_t* nbr, float* t_out, int32_t* eid_out, void* ws, size_t ws_bytes,
                            hipStream_t s);

// attention
// Fused merge-layer chains (merge.hip): float32 and the attention / memory widths they are built for.
bool merge_fused_ok(int dtype, int da, int dm);
size_t merge_weights_floats(int da, int dm, int dt);
// dst[rows x cols] (contiguous): dst[r][c] = src[r * ld + c] (tr: src[c * ld + r]) for r < n, c < k, else 0.
// ldd: the destination's row stride (0: cols).
struct PadCopy {
  const float* src;
  float* dst;
  int rows, cols, n, k, ld, tr, ldd;
};
inline PadCopy plain_copy(const float* src, float* dst, int rows, int cols) {
  return PadCopy{src, dst, rows, cols, rows, cols, cols, 0, 0};
}
// The four copies of link_prepare_weights as descriptors (4 written to out), or 0 at widths the fused
// decoder does not take.
int link_pad_copies(const float* W1, int da, float* Wp, PadCopy* out);
// Zero-padded copies in one launch (n <= 18).
mtgnn_status pad_copies(const PadCopy* c, int n, hipStream_t s);
// The fused decoder's weight copies in the link workspace (nothing at the general widths): as
// descriptors (returns how many, 0 or 4), or made on s.
int link_copies_impl(const mtgnn_link_params* p, const mtgnn_dims* d, int64_t max_q, void* ws, PadCopy* out);
mtgnn_status link_prepare_impl(const mtgnn_link_params* p, const mtgnn_dims* d, int64_t max_q, void* ws,
                               hipStream_t s);
// The zero-padded copies of W_d1's two column halves and their transposes that link_fused reads from Wp.
mtgnn_status link_prepare_weights(const float* W1, int da, float* Wp, hipStream_t s);
// The query projection's constant: out[j] = bq[j] + sum_t Wq[j][dm + t] cos(w_t 0 + b_t) (a query's
// time input is phi(0)); Wq row stride dm + dt.
struct QConst {
  const float *Wq, *bq, *tw, *tb;
  float* out;
  int da, dm, dt;
};
// One launch: the padded merge copies, then the extra copies (at most eight), and the query constant
// when qc is given.
mtgnn_status merge_prepare(const float* Wo, const float* W1, const float* W2, int da, int dm, float* Wp,
                           hipStream_t s, const PadCopy* extra = nullptr, int n_extra = 0,
                           const QConst* qc = nullptr);
// The query projection on the same machinery (float32, the widths qproj_fused_ok accepts); its padded
// copies (qproj_copy 0: W_q[:, :dm], 1: W_q[:, :dm]^T) follow the merge copies in the same buffer.
bool qproj_fused_ok(int dtype, int da, int dm, int dt);
PadCopy qproj_copy(const float* Wq, int da, int dm, int dt, float* Wp, int which);
// qv = W_q[:, :dm] q_in[:, :dm] + cq, cq = b_q + W_q[:, dm:] phi(0) (QConst): a query's time input is
// the constant phi(0).
mtgnn_status qproj_fwd_fused(const float* q_in, const float* Wp, const float* cq, float* qv, const int32_t* n_q,
                             int64_t max_q, int da, int dm, int dt, hipStream_t s);
mtgnn_status qproj_dx_fused(const float* dqv, const float* Wp, float* dm_in, int64_t ldm, const int32_t* n_q,
                            int64_t max_q, int da, int dm, int dt, hipStream_t s);
// The d M' product (d_mem += S[:, dm:] W_kv[:, :dm]) on the same machinery, for the shapes qproj_fused_ok
// accepts; dmem_copy 0 / 1 are its padded weight's two halves (from W_k, from W_v).
PadCopy dmem_copy(const float* Wk, const float* Wv, int da, int dm, int dt, int Dkv, float* Wp, int which);
// The GRU backward's time-feature gradient on the same machinery (float32; gru_dx_fused_ok shapes), from
// W_ih[:, 2 dm : 2 dm + dt]^T zero-padded to gru_dx_weight_floats floats (written by the GRU update).
bool gru_dx_fused_ok(int dtype, int dm, int dt);
size_t gru_dx_weight_floats(int dm, int dt);
mtgnn_status gru_dx_fused(const float* dgi, const float* WT, float* dmsg_time, const int32_t* n_rows,
                          int64_t max_rows, int dm, int dt, hipStream_t s);
mtgnn_status dmem_dx_fused(const float* S, int64_t ldS, const float* Wp, float* d_mem, const int32_t* n_rows,
                           int64_t max_rows, int da, int dm, int dt, hipStream_t s);
mtgnn_status merge_fwd_fused(const float* attn, float* m_in, const float* Wp, const float* bo, const float* b1,
                             const float* b2, float* m1, float* a1, float* z, const int32_t* n_q, int64_t max_q,
                             int da, int dm, hipStream_t s);
mtgnn_status merge_bwd_fused(const float* dz, const float* Wp, const float* m1, float* dm1, float* dm_in,
                             float* dattn, const int32_t* n_q, int64_t max_q, int da, int dm, hipStream_t s);

size_t attn_save_bytes(const mtgnn_dims* d, int64_t max_q);
size_t attn_fwd_ws(const mtgnn_dims* d, int64_t max_q);
mtgnn_status attn_fwd_impl(const int32_t* q_node, const float* q_t, const int32_t* n_q, int64_t max_q,
                           const int32_t* nbr, const float* nt, const int32_t* neid, const void* memory,
                           const float* edge_feat, const float* tw, const float* tb, const mtgnn_attn_params* p,
                           const mtgnn_dims* d, float* z, void* save, void* ws, size_t ws_bytes, hipStream_t s);
// The forward's inputs that need only the sampled neighbours and the weights (stacked key/value
// weights, padded merge weights, per-query valid-slot counts and offsets), then the rest.
// more, n_more: up to 4 further zero-padded copies, made in the same launch on the float32 fused path.
mtgnn_status attn_prepare_weights_impl(const mtgnn_attn_params* p, const float* tw, const float* tb,
                                       const mtgnn_dims* d, void* save, hipStream_t s,
                                       const PadCopy* more = nullptr, int n_more = 0);
mtgnn_status attn_prepare_slots_impl(const int32_t* nbr, const int32_t* n_q, int64_t max_q, const mtgnn_dims* d,
                                     void* save, void* ws, size_t ws_bytes, hipStream_t s);
mtgnn_status attn_prepare_impl(const int32_t* nbr, const int32_t* n_q, int64_t max_q, const mtgnn_attn_params* p,
                               const float* tw, const float* tb, const mtgnn_dims* d, void* save, void* ws,
                               size_t ws_bytes, hipStream_t s);
mtgnn_status attn_fwd_prepared_impl(const int32_t* q_node, const float* q_t, const int32_t* n_q, int64_t max_q,
                                    const int32_t* nbr, const float* nt, const int32_t* neid, const void* memory,
                                    const float* edge_feat, const float* tw, const float* tb,
                                    const mtgnn_attn_params* p, const mtgnn_dims* d, float* z, void* save,
                                    hipStream_t s);
size_t attn_bwd_ws(const mtgnn_dims* d, int64_t max_q, int64_t max_rows);
mtgnn_status attn_bwd_impl(const int32_t* q_node, const float* q_t, const int32_t* n_q, int64_t max_q,
                           const int32_t* nbr, const float* nt, const float* dz, const void* save, const int32_t* uniq,
                           const int32_t* n_rows, int64_t max_rows, const float* tw, const float* tb,
                           const mtgnn_attn_params* p, const mtgnn_dims* d, mtgnn_attn_grads* g, float* d_mem,
                           float* d_time_w, float* d_time_b, void* ws, size_t ws_bytes, hipStream_t s,
                           hipStream_t s_dmem = nullptr, hipEvent_t fork = nullptr, hipEvent_t join = nullptr,
                           bool grouped = false);
// The backward's d M' grouping alone (row map, occurrence keys, stable sort, segment bounds) into ws,
// from the queries, the sampled neighbours, the slot counts in save and the updated rows.
mtgnn_status attn_bwd_group_impl(const int32_t* q_node, const int32_t* n_q, int64_t max_q, const int32_t* nbr,
                                 const void* save, const int32_t* uniq, const int32_t* n_rows, int64_t max_rows,
                                 const mtgnn_dims* d, void* ws, size_t ws_bytes, hipStream_t s);

}  // namespace mtgnn

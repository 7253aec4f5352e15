/*
 * mtgnn -- the single-GPU batch step of memory-based temporal GNN training
 * (TGN-style memory + temporal attention) for AMD Instinct MI355X (gfx950).
 *
 * The paper this implements (DepTGL, arXiv 2608.16305) describes distributed
 * training of memory-based TGNNs.  Each worker executes mixed batches of target
 * events and replayed auxiliary events (Definition 2, Eq. 5), with load-aware
 * pruning of replay events (Eq. 10-11) and a loss masked to target events
 * (Eq. 12-13).  Inside a batch the model follows the chronological node-state
 * semantics of Section III-A (Eq. 1-2).  This library is that per-worker
 * hot path on one GPU.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Every pointer argument named as device data points to device memory owned
 *   by the caller.  The library never allocates, frees or synchronises, except
 *   where an entry point says so.  Each call only enqueues kernels on `stream`
 *   and returns; results are ready when the stream reaches them.
 * - Scratch memory is passed as (ws, ws_bytes).  The required size comes from
 *   mtgnn_workspace_bytes(); a smaller workspace returns MTGNN_EWORKSPACE.
 *   Workspace contents need not be initialised and are garbage afterwards.
 *   Calls that run at the same time need separate workspaces.
 * - Arguments are validated on the host before any HIP call:
 *   - null required pointers, non-positive sizes or an inconsistent
 *     mtgnn_dims give MTGNN_EINVAL;
 *   - an unknown dtype gives MTGNN_EUNSUPPORTED;
 *   - a failed kernel launch gives MTGNN_EHIP (the HIP message is kept for
 *     mtgnn_last_error()).
 *   Device-resident preconditions are documented per call and are not checked.
 *   These are index ranges, the event order and finite timestamps.
 * - Device-side counts (`n_rows`, `n_q`, ...) are single int32 values in device
 *   memory written by an earlier call.  The host passes the matching maximum
 *   (`max_rows`, `max_q`), which sizes the buffers and grids.  A NULL count
 *   means the maximum is exact.
 * - Matrices are row-major.  Weights use the [out, in] layout of a linear
 *   layer, y = x W^T + b.  Weights and the memory table are stored in the
 *   dims' dtype: float32, or bfloat16 bit patterns rounded to nearest even.
 *   Biases, timestamps, the time encoder and every gradient are float32.
 * - Memory rows are dense: row n of the table starts at element n * d_mem.
 */
#ifndef MTGNN_H
#define MTGNN_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MTGNN_OK = 0,
  MTGNN_EINVAL = -1,
  MTGNN_EUNSUPPORTED = -2,
  MTGNN_EWORKSPACE = -3,
  MTGNN_EHIP = -4
} mtgnn_status;

typedef enum { MTGNN_F32 = 0, MTGNN_BF16 = 1 } mtgnn_dtype;

/* Model and table sizes.  d_msg = 2 d_mem + d_time + d_edge is the message width,
 * d_kv = d_mem + d_edge + d_time the key/value input width, d_q = d_mem + d_time the
 * query input width.  n_heads must divide d_attn.  d_edge may be 0. */
typedef struct {
  int64_t n_nodes;
  int32_t d_mem, d_time, d_edge, d_attn, n_heads, k;
  int32_t dtype; /* mtgnn_dtype */
} mtgnn_dims;

/* One mixed batch (Definition 2, Eq. 5), as device arrays of length n.
 *   src, dst -- event endpoints u_k, v_k (Section III-A), node ids in [0, n_nodes);
 *   t        -- timestamps, float32;
 *   eid      -- event ids, which index the edge-feature rows;
 *   flags    -- event-type mask, or NULL when every event is a target:
 *               bit 0 = replayed auxiliary event (no query, no loss);
 *               bit 1 = pruned by load-aware pruning (Eq. 10-11).
 * Precondition: events are sorted by (t, eid) ascending and eids are unique. */
typedef struct {
  int64_t n;
  const int32_t* src;
  const int32_t* dst;
  const int32_t* eid;
  const float* t;
  const uint8_t* flags;
} mtgnn_batch;

/* Attention parameters.  Weights are in the dims' dtype, biases are float32.
 *   W_q [d_attn, d_q], W_k and W_v [d_attn, d_kv], W_o [d_attn, d_attn],
 *   W_1 [d_attn, d_attn + d_mem], W_2 [d_attn, d_attn]. */
typedef struct {
  const void *W_q, *W_k, *W_v, *W_o, *W_1, *W_2;
  const float *b_q, *b_k, *b_v, *b_o, *b_1, *b_2;
} mtgnn_attn_params;

/* Link-prediction decoder parameters (float32 whatever the dims' dtype): the edge score
 *   s(a, b) = W_d2 relu(W_d1 [z_a || z_b] + b_d1) + b_d2,
 * W_d1 [d_attn, 2 d_attn], b_d1 [d_attn], W_d2 [1, d_attn], b_d2 [1]. */
typedef struct {
  const float *W_d1, *b_d1, *W_d2, *b_d2;
} mtgnn_link_params;

/* Decoder parameter gradients (float32, same shapes, overwritten). */
typedef struct {
  float *W_d1, *b_d1, *W_d2, *b_d2;
} mtgnn_link_grads;

/* Attention parameter gradients (float32, same shapes, overwritten). */
typedef struct {
  float *W_q, *W_k, *W_v, *W_o, *W_1, *W_2;
  float *b_q, *b_k, *b_v, *b_o, *b_1, *b_2;
} mtgnn_attn_grads;

typedef enum {
  MTGNN_OP_BUILD_QUERIES = 0,
  MTGNN_OP_AGGREGATE_LAST = 1,
  MTGNN_OP_BUILD_MESSAGES = 2,
  MTGNN_OP_GRU_UPDATE = 3,
  MTGNN_OP_SAMPLE_RECENT = 4,
  MTGNN_OP_TEMPORAL_ATTN = 5,
  MTGNN_OP_TEMPORAL_ATTN_BWD = 6,
  MTGNN_OP_GRU_UPDATE_BWD = 7,
  MTGNN_OP_BUILD_MESSAGES_BWD = 8,
  MTGNN_OP_BUILD_CSR = 9,
  MTGNN_OP_LINK_LOSS = 10,
  MTGNN_OP_MIXED_BATCHES = 11,
  MTGNN_OP_RNN_UPDATE = 12,
  MTGNN_OP_RNN_UPDATE_BWD = 13,
  MTGNN_OP_TIME_PROJECTION_BWD = 14
} mtgnn_op;

/* Workspace bytes for `op`.  max_rows is the batch size n for BUILD_QUERIES and
 * AGGREGATE_LAST, the row maximum for the memory-phase ops, and the number of
 * stream events for BUILD_CSR.  max_q is the query maximum for the attention
 * ops.  Unused sizes are ignored.  Returns 0 for an invalid request. */
size_t mtgnn_workspace_bytes(int op, const mtgnn_dims* dims, int64_t max_rows, int64_t max_q);

/* Bytes of the forward save buffer that the backward call of `op` reads.
 * op = MTGNN_OP_GRU_UPDATE, MTGNN_OP_RNN_UPDATE or MTGNN_OP_TEMPORAL_ATTN; 0 otherwise. */
size_t mtgnn_save_bytes(int op, const mtgnn_dims* dims, int64_t max_rows, int64_t max_q);

/* Batch intake (Definition 2 and Eq. 12).  Builds the query list of
 * the target events (flags & 3 == 0) in batch order as three blocks:
 * sources, then destinations, then negatives, each at its event's time.
 *   neg    -- [b->n] negative destination per event (device);
 *   q_node -- [3 b->n] out; q_t -- [3 b->n] out;
 *   n_q    -- device int32 out = 3 * (number of target events).
 * Entries at or beyond n_q are left untouched. */
mtgnn_status mtgnn_build_queries(const mtgnn_batch* b, const int32_t* neg, int32_t* q_node, float* q_t,
                                 int32_t* n_q, void* ws, size_t ws_bytes, hipStream_t stream);

/* Most-recent message aggregation (Eq. 2 applied once per batch; TGN's last-message aggregator,
 * Section VII-A).
 * Every non-pruned event i sends message 2i to src[i] (role 0) and message
 * 2i+1 to dst[i] (role 1).  For each node that receives a message, the winner
 * is its message with the largest (t, eid, role).  Under the batch order
 * precondition that is the largest message index; a self-loop's role 1 wins.
 *   uniq   -- [2 b->n] out: receiving nodes, one row each, in increasing order
 *             of their winning message (the order of each node's last message
 *             in the batch);
 *   winner -- [2 b->n] out: winner message index (2i + role) per uniq entry,
 *             so winner[0 .. n_uniq) is strictly increasing;
 *   n_uniq -- device int32 out: number of entries written.
 * The workspace holds an n_nodes-entry node table (no initialisation needed).
 * Integer-exact and deterministic: integer max per node, fixed-order compaction. */
mtgnn_status mtgnn_aggregate_last(const mtgnn_batch* b, int64_t n_nodes, int32_t* uniq, int32_t* winner,
                                  int32_t* n_uniq, void* ws, size_t ws_bytes, hipStream_t stream);

/* Message construction (Eq. 1) for each aggregated row r < n_rows.
 * Let i = winner[r] / 2 be the event, node = uniq[r] and partner its other
 * endpoint.  Then
 *     msg[r] = [ M[node] || M[partner] || cos(time_w * dt + time_b) || x[eid_i] ],
 *     dt[r]  = t_i - last_update[node].
 * dt is a float32 subtraction.  The cosine argument rounds the product and
 * then the sum to float32, with no fused multiply-add.
 *   memory      -- [n_nodes, d_mem] (dtype); last_update [n_nodes] float32;
 *   edge_feat   -- [*, d_edge] float32 indexed by eid (NULL iff d_edge == 0);
 *   time_w, time_b -- [d_time] float32;
 *   msg         -- [max_rows, d_msg] out (dtype); dt -- [max_rows] float32 out.
 * Reads only the pre-update table, so call it before mtgnn_gru_update. */
mtgnn_status mtgnn_build_messages(const mtgnn_batch* b, const int32_t* uniq, const int32_t* winner,
                                  const int32_t* n_rows, int64_t max_rows, const void* memory,
                                  const float* last_update, const float* edge_feat, const float* time_w,
                                  const float* time_b, const mtgnn_dims* dims, void* msg, float* dt,
                                  hipStream_t stream);

/* GRU memory update (Eq. 2; TGN's memory updater, Section VII-A), gate order r, z, n:
 *   r = sig(W_ir x + b_ir + W_hr h + b_hr),  z = sig(W_iz x + b_iz + W_hz h + b_hz),
 *   n = tanh(W_in x + b_in + r * (W_hn h + b_hn)),  h' = (1 - z) n + z h,
 * with x = msg[r] and h = memory[uniq[r]].  Writes memory[uniq[r]] = h'
 * (rounded to the dtype) and last_update[uniq[r]] = t of the winning event.
 * Rows not in uniq are never touched.
 *   W_ih [3 d_mem, d_msg], W_hh [3 d_mem, d_mem] (dtype); b_ih, b_hh [3 d_mem] float32;
 *   save -- mtgnn_save_bytes(MTGNN_OP_GRU_UPDATE) bytes for the backward, or NULL. */
mtgnn_status mtgnn_gru_update(const mtgnn_batch* b, const int32_t* uniq, const int32_t* winner,
                              const int32_t* n_rows, int64_t max_rows, const void* msg, const void* W_ih,
                              const void* W_hh, const float* b_ih, const float* b_hh, const mtgnn_dims* dims,
                              void* memory, float* last_update, void* save, void* ws, size_t ws_bytes,
                              hipStream_t stream);

/* Most-recent-k temporal neighbour sampling over the temporal adjacency: the
 * temporal neighbourhood that TGN aggregates (Section VII-A), strictly before the
 * query time so that an event never sees itself or later events (Section III-A).
 * The adjacency holds every stream event in both directions.
 * For query (n, tau), take the entries of node n with t < tau (strictly),
 * then the k largest by (t, eid, role), newest first.  Missing slots are
 * padded with nbr = -1, t = 0, eid = -1.
 *   csr_off [n_nodes+1] int64; csr_nbr, csr_eid int32 and csr_t float32 [2E],
 *     each node's entries sorted by (t, eid, role) ascending
 *     (as mtgnn_build_temporal_csr writes them);
 *   q_node, q_t [max_q]; out_nbr, out_t, out_eid [max_q, k] out.
 * Integer-exact. */
mtgnn_status mtgnn_sample_recent(const int64_t* csr_off, const int32_t* csr_nbr, const float* csr_t,
                                 const int32_t* csr_eid, int64_t n_nodes, const int32_t* q_node,
                                 const float* q_t, const int32_t* n_q, int64_t max_q, int32_t k,
                                 int32_t* out_nbr, float* out_t, int32_t* out_eid, hipStream_t stream);

/* One-layer multi-head temporal attention embedding (TGN's temporal neighbourhood
 * aggregation, Section VII-A), for each query q.
 *   q     = W_q [M[q_node] || phi(0)] + b_q
 *   K_j   = W_k [M[nbr_j] || x[eid_j] || phi(q_t - t_j)] + b_k,  V_j likewise with W_v
 *   per head h (d_attn / n_heads columns), over valid slots j (nbr_j >= 0):
 *     p = softmax_j(q_h . K_jh / sqrt(d_attn / n_heads)),  a_h = sum_j p_j V_jh
 *     (a = 0 when no slot is valid)
 *   o     = W_o a + b_o
 *   z     = W_2 relu(W_1 [o || M[q_node]] + b_1) + b_2
 * phi(dt) = cos(time_w * dt + time_b) with the rounding of mtgnn_build_messages.
 *   nbr, nt, neid -- [max_q, k] as written by mtgnn_sample_recent;
 *   memory        -- the table after this step's mtgnn_gru_update;
 *   z             -- [max_q, d_attn] float32 out;
 *   save          -- mtgnn_save_bytes(MTGNN_OP_TEMPORAL_ATTN) bytes for the backward. */
mtgnn_status mtgnn_temporal_attn(const int32_t* q_node, const float* q_t, const int32_t* n_q, int64_t max_q,
                                 const int32_t* nbr, const float* nt, const int32_t* neid, const void* memory,
                                 const float* edge_feat, const float* time_w, const float* time_b,
                                 const mtgnn_attn_params* params, const mtgnn_dims* dims, float* z, void* save,
                                 void* ws, size_t ws_bytes, hipStream_t stream);

/* The attention embedding in two calls, for callers that run the first on another stream while
 * the memory table is still being updated (it reads neither the memory nor
 * the queries).  mtgnn_temporal_attn is exactly
 * mtgnn_temporal_attn_prepare followed by mtgnn_temporal_attn_prepared on
 * one stream, and the results are bitwise the same.
 *   _prepare  -- from nbr (valid slots lead each row) and the weights, writes
 *                into save the stacked [W_k; W_v] and [b_k; b_v], the padded
 *merge-layer weights (float32), the query projection's constant
 *                term b_q + W_q[:, d_mem:] cos(time_b) (every query's time
 *                input is the encoding of 0, so its share is one vector; it
 *                needs time_w and time_b, the forward's) and the per-query
 *                valid-slot counts, their exclusive prefix sums and the
 *                valid total; ws as for mtgnn_temporal_attn.  It is exactly
 *                _prepare_weights (the weight copies and that constant: they
 *                read only the parameters, and their place in save does not
 *                depend on max_q)
 *                followed by _prepare_slots (the counts, offsets and total);
 *                the two may run on different streams, in either order.
 *   _prepared -- the rest of the forward, reading what _prepare wrote into
 *                the same save (same nbr, n_q, max_q, weights and dims); the
 *                caller orders it after _prepare (same stream, or an event).
 * Arguments, layouts and errors as for mtgnn_temporal_attn. */
mtgnn_status mtgnn_temporal_attn_prepare(const int32_t* nbr, const int32_t* n_q, int64_t max_q,
                                         const mtgnn_attn_params* params, const float* time_w, const float* time_b,
                                         const mtgnn_dims* d, void* save, void* ws, size_t ws_bytes,
                                         hipStream_t stream);
mtgnn_status mtgnn_temporal_attn_prepare_weights(const mtgnn_attn_params* params, const float* time_w,
                                                 const float* time_b, const mtgnn_dims* d, void* save,
                                                 hipStream_t stream);
mtgnn_status mtgnn_temporal_attn_prepare_slots(const int32_t* nbr, const int32_t* n_q, int64_t max_q,
                                               const mtgnn_dims* d, void* save, void* ws, size_t ws_bytes,
                                               hipStream_t stream);
mtgnn_status mtgnn_temporal_attn_prepared(const int32_t* q_node, const float* q_t, const int32_t* n_q, int64_t max_q,
                                          const int32_t* nbr, const float* nt, const int32_t* neid,
                                          const void* memory, const float* edge_feat, const float* time_w,
                                          const float* time_b, const mtgnn_attn_params* params, const mtgnn_dims* d,
                                          float* z, void* save, hipStream_t stream);

/* Backward of the attention embedding, mtgnn_temporal_attn for the output gradient dz [max_q, d_attn].
 * The caller computes dz from the masked loss (Eq. 13).
 *   grads -- every attention parameter gradient (overwritten);
 *   d_mem -- [max_rows, d_mem] float32 out, row r aligned with uniq[r]: the sum of
 *            the gradients of every occurrence of node uniq[r], as a query or as a
 *            valid neighbour.  Memory rows not in uniq get no gradient, because the
 *            table is not differentiated across steps;
 *   d_time_w, d_time_b -- [d_time] float32, OVERWRITTEN with the attention's share of the
 *            time-encoder gradient (mtgnn_build_messages_bwd then adds the messages' share).
 * q_node ... neid, memory, edge_feat and save are the forward call's.
 * uniq/n_rows are the rows updated by this step's memory phase (mtgnn_aggregate_last). */
mtgnn_status mtgnn_temporal_attn_bwd(const int32_t* q_node, const float* q_t, const int32_t* n_q, int64_t max_q,
                                     const int32_t* nbr, const float* nt, const float* dz, const void* save,
                                     const int32_t* uniq, const int32_t* n_rows, int64_t max_rows,
                                     const float* time_w, const float* time_b, const mtgnn_attn_params* params,
                                     const mtgnn_dims* dims, mtgnn_attn_grads* grads, float* d_mem,
                                     float* d_time_w, float* d_time_b, void* ws, size_t ws_bytes,
                                     hipStream_t stream);

/* Attention backward with two streams: the same computation, arguments and results as
 * mtgnn_temporal_attn_bwd, with the d_mem part (grouping every occurrence of
 * an updated node and summing it) enqueued on a second stream so that it runs
 * concurrently with the parameter gradients, which stay on `stream`.
 *   dmem_stream -- a second stream of the caller, at the default priority;
 *   fork, join  -- two events of the caller (timing may be disabled).
 * The call records `fork` on `stream` at entry and makes dmem_stream wait for
 * it (the grouping's key sort, which reads only forward outputs, starts there
 * while the data gradients run on `stream`), records `fork` again once the
 * gradients the sums need are ready and makes dmem_stream wait for it (the
 * sums), records `join` on dmem_stream and makes `stream` wait for `join`:
 * work enqueued on `stream` afterwards is ordered after both parts, as with
 * mtgnn_temporal_attn_bwd.  Results are bitwise identical to it.  The two
 * parts use disjoint regions of ws (the same size as for
 * mtgnn_temporal_attn_bwd).  Errors: as mtgnn_temporal_attn_bwd; EINVAL if
 * dmem_stream, fork or join is NULL while max_rows > 0. */
mtgnn_status mtgnn_temporal_attn_bwd_overlap(const int32_t* q_node, const float* q_t, const int32_t* n_q,
                                             int64_t max_q, const int32_t* nbr, const float* nt, const float* dz,
                                             const void* save, const int32_t* uniq, const int32_t* n_rows,
                                             int64_t max_rows, const float* time_w, const float* time_b,
                                             const mtgnn_attn_params* params, const mtgnn_dims* dims,
                                             mtgnn_attn_grads* grads, float* d_mem, float* d_time_w,
                                             float* d_time_b, void* ws, size_t ws_bytes, hipStream_t stream,
                                             hipStream_t dmem_stream, hipEvent_t fork, hipEvent_t join);

/* Attention backward, the d_mem grouping ahead of the gradients: every occurrence of an updated node among the
 * queries and the valid neighbour slots, keyed by its updated row, sorted stably by key, and each
 * row's segment bounds, written into ws (the backward's workspace, mtgnn_workspace_bytes for
 * MTGNN_OP_TEMPORAL_ATTN_BWD).  It reads only q_node / n_q, the sampled neighbours nbr
 * [max_q, k], the slot counts and offsets that the attention's preparation left in save, and the
 * updated rows uniq / n_rows, so it may run before the forward's gather and long before any
 * gradient exists; the caller runs it on the stream it will pass as dmem_stream to
 * mtgnn_temporal_attn_bwd_grouped, which consumes it.  Between the two calls nothing may write
 * ws, save's slot counts, uniq or n_rows.  max_rows == 0: nothing to do.  Errors: EINVAL (a NULL
 * pointer, max_q out of range), EWORKSPACE. */
mtgnn_status mtgnn_temporal_attn_bwd_group(const int32_t* q_node, const int32_t* n_q, int64_t max_q,
                                           const int32_t* nbr, const void* save, const int32_t* uniq,
                                           const int32_t* n_rows, int64_t max_rows, const mtgnn_dims* dims,
                                           void* ws, size_t ws_bytes, hipStream_t stream);

/* Attention backward with two streams, the grouping done ahead: as mtgnn_temporal_attn_bwd_overlap, except that
 * the d_mem grouping is the one mtgnn_temporal_attn_bwd_group left in ws, so there is no fork at
 * entry.  dmem_stream must be ordered after that call (it was enqueued on dmem_stream, or
 * dmem_stream waits for it).  The call records `fork` on `stream` once the gradients the sums need
 * are ready, makes dmem_stream wait for it (the sums), records `join` on dmem_stream and makes
 * `stream` wait for `join`.  join may be NULL: then the call records and waits for nothing at the
 * end, and the caller must order later work on `stream` after dmem_stream itself (an event recorded
 * on dmem_stream after its own later work there serves).  Results are bitwise identical to
 * mtgnn_temporal_attn_bwd.  Errors: as mtgnn_temporal_attn_bwd_overlap; EINVAL if dmem_stream or
 * fork is NULL while max_rows > 0. */
mtgnn_status mtgnn_temporal_attn_bwd_grouped(const int32_t* q_node, const float* q_t, const int32_t* n_q,
                                             int64_t max_q, const int32_t* nbr, const float* nt, const float* dz,
                                             const void* save, const int32_t* uniq, const int32_t* n_rows,
                                             int64_t max_rows, const float* time_w, const float* time_b,
                                             const mtgnn_attn_params* params, const mtgnn_dims* dims,
                                             mtgnn_attn_grads* grads, float* d_mem, float* d_time_w,
                                             float* d_time_b, void* ws, size_t ws_bytes, hipStream_t stream,
                                             hipStream_t dmem_stream, hipEvent_t fork, hipEvent_t join);

/* The masked batch loss of Eq. 13 with the link-prediction edge loss, and its gradient.
 * z holds the embeddings of the batch's queries as mtgnn_build_queries lists them: the src of
 * the n_tar target events, then their dst, then their negatives, n_tar = n_q / 3 (replayed
 * and pruned events have no query: this is the target mask M_p of Eq. 12).  Each target
 * event's edge loss is the binary cross-entropy of its true edge (label 1) and its negative
 * edge (label 0) under the decoder score s that mtgnn_link_params defines, TGN's link predictor
 * (Section VII-A):
 *   l = softplus(-s(src, dst)) + softplus(s(src, neg)),
 * and the batch loss is the mean of l over the target events, or 0 when there is none.
 *   z      -- [max_q, d_attn] float32 (mtgnn_temporal_attn's output); max_q a multiple of 3;
 *   loss   -- device float32 scalar out;
 *   scores -- [2, max_q / 3] float32 out, s(src, dst) then s(src, neg) per target event, or NULL;
 *   dz     -- [max_q, d_attn] float32 out: d loss / d z, rows < n_q (the input of
 *             mtgnn_temporal_attn_bwd);
 *   grads  -- the decoder's gradients, overwritten (zero when there is no target event).
 * Deterministic: every sum runs in a fixed order.  Errors: EINVAL (NULL pointers, max_q not a
 * multiple of 3), EUNSUPPORTED (d_attn > 128), EWORKSPACE. */
mtgnn_status mtgnn_link_loss(const float* z, const int32_t* n_q, int64_t max_q, const mtgnn_link_params* params,
                             const mtgnn_dims* dims, float* loss, float* scores, float* dz, mtgnn_link_grads* grads,
                             void* ws, size_t ws_bytes, hipStream_t stream);

/* The masked batch loss with its last reductions and the decoder's first-layer weight gradient on a
 * second stream: the same computation, arguments and results as mtgnn_link_loss (bitwise), except that
 * once scores, dz and the per-block partial sums are enqueued on `stream`, the call records `fork` on
 * `stream`, makes dw_stream wait for it and enqueues the loss, grads->W_d2, grads->b_d2, grads->W_d1 and
 * grads->b_d1 on dw_stream (for the widths the fused decoder kernel takes: d_attn a multiple of 4 in
 * 17..32 or 97..112; at other widths everything runs on `stream` and nothing is recorded).  Work
 * enqueued on `stream` afterwards (the attention backward, which needs only dz) overlaps it.  The loss
 * and the decoder's gradients are complete when the work this call enqueued on dw_stream is; until
 * then the caller writes neither z nor ws and reads neither the loss nor those gradients (an event
 * recorded on dw_stream after this call, or later work on dw_stream, orders that).
 *   dw_stream -- a second stream of the caller, at the default priority;
 *   fork      -- an event of the caller (timing may be disabled).
 * Errors: as mtgnn_link_loss; EINVAL if dw_stream or fork is NULL; EHIP if the fork cannot be recorded
 * or waited for. */
mtgnn_status mtgnn_link_loss_overlap(const float* z, const int32_t* n_q, int64_t max_q,
                                     const mtgnn_link_params* params, const mtgnn_dims* dims, float* loss,
                                     float* scores, float* dz, mtgnn_link_grads* grads, void* ws, size_t ws_bytes,
                                     hipStream_t stream, hipStream_t dw_stream, hipEvent_t fork);

/* The decoder's weight copies of mtgnn_link_loss (Eq. 13's scoring layer), made ahead on any stream so
 * that the loss itself need not make them: the zero-padded column halves of params->W_d1 and their
 * transposes, written into ws (the workspace a later mtgnn_link_loss_prepared call with the same
 * d_attn and max_q gets; nothing else in ws is touched).  At widths the fused decoder kernel does not
 * take (d_attn a multiple of 4 in 17..32 or 97..112) nothing is written.  The copies stay valid until
 * W_d1 or ws is written again.
 * Errors: as mtgnn_link_loss for max_q, dims, params->W_d1 and ws. */
mtgnn_status mtgnn_link_prepare_weights(const mtgnn_link_params* params, const mtgnn_dims* dims, int64_t max_q,
                                        void* ws, size_t ws_bytes, hipStream_t stream);

/* mtgnn_temporal_attn_prepare_weights and mtgnn_link_prepare_weights (link, max_q, link_ws) in one
 * call: for float32 weights of the fused merge and decoder widths, every copy of both is made by a
 * single launch.  Arguments, results and errors as those two calls. */
mtgnn_status mtgnn_temporal_attn_prepare_weights_link(const mtgnn_attn_params* params, const float* time_w,
                                                      const float* time_b, const mtgnn_dims* dims, void* save,
                                                      const mtgnn_link_params* link, int64_t max_q, void* link_ws,
                                                      size_t link_ws_bytes, hipStream_t stream);

/* mtgnn_link_loss (dw_stream and fork NULL) or mtgnn_link_loss_overlap (both given) with the decoder's
 * weight copies already in ws: a mtgnn_link_prepare_weights call with the same params->W_d1, dims,
 * max_q and ws, ordered before this call on `stream` (same stream, or an event the caller records
 * after it and `stream` waits for), and W_d1 not written since.  Same computation and bitwise results
 * as those calls.  Errors: as mtgnn_link_loss_overlap; EINVAL if only one of dw_stream and fork is
 * NULL. */
mtgnn_status mtgnn_link_loss_prepared(const float* z, const int32_t* n_q, int64_t max_q,
                                      const mtgnn_link_params* params, const mtgnn_dims* dims, float* loss,
                                      float* scores, float* dz, mtgnn_link_grads* grads, void* ws, size_t ws_bytes,
                                      hipStream_t stream, hipStream_t dw_stream, hipEvent_t fork);

/* Backward of the GRU memory update (Eq. 2), mtgnn_gru_update, for d_mem = dL/dh' [max_rows, d_mem].
 * The previous memory h is detached.
 *   save, msg   -- the forward call's (save must not be NULL there);
 *   dW_ih, dW_hh, db_ih, db_hh -- float32, overwritten;
 *   dmsg_time   -- [max_rows, d_time] float32 out: dL/dphi for the message time slice,
 *                  the only message slice the step back-propagates (memory and edge
 *                  features are inputs, not parameters). */
mtgnn_status mtgnn_gru_update_bwd(const float* d_mem, const void* save, const void* msg, const int32_t* n_rows,
                                  int64_t max_rows, const void* W_ih, const void* W_hh, const mtgnn_dims* dims,
                                  float* dW_ih, float* dW_hh, float* db_ih, float* db_hh, float* dmsg_time,
                                  void* ws, size_t ws_bytes, hipStream_t stream);

/* Time-encoder gradient of the messages (Eq. 1), ACCUMULATED into d_time_w/d_time_b:
 *   d_time_w[j] += sum_r dmsg_time[r, j] * (-sin(arg_rj)) * dt[r]
 *   d_time_b[j] += sum_r dmsg_time[r, j] * (-sin(arg_rj))
 * where arg_rj = time_w[j] * dt[r] + time_b[j], rounded as in mtgnn_build_messages.
 * Reductions run in a fixed order (deterministic). */
mtgnn_status mtgnn_build_messages_bwd(const float* dmsg_time, const float* dt, const int32_t* n_rows,
                                      int64_t max_rows, const float* time_w, const float* time_b,
                                      const mtgnn_dims* dims, float* d_time_w, float* d_time_b, void* ws,
                                      size_t ws_bytes, hipStream_t stream);

/* mtgnn_build_messages_bwd without a workspace, for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc).  Same arguments, computation,
 * kernels and bitwise results as mtgnn_build_messages_bwd, minus (ws, ws_bytes): the row-chunk partial
 * sums live in a device scratch array of MTGNN_NOALLOC_SCRATCH_BYTES (4 MiB) that the library holds on
 * every GPU it runs on until the process ends.  The call allocates and frees nothing.
 *   - The request needs 8 * d_time * ceil(max_rows / 32) bytes (rounded up to 256); beyond 4 MiB the
 *     call returns MTGNN_EWORKSPACE before any launch (d_time = 100 allows max_rows up to 167,744).
 *   - `stream` must belong to the current device (else MTGNN_EINVAL); its first call on a device looks
 *     up that device's scratch address (MTGNN_EHIP if that fails).
 *   - Every call on one GPU shares that GPU's scratch, which keeps the last call's partials (nothing in
 *     it needs to start at zero).  Calls that overlap on one GPU (other streams, other host threads)
 *     race on it: order them. */
#define MTGNN_NOALLOC_SCRATCH_BYTES (4 << 20)
mtgnn_status mtgnn_build_messages_bwd_noalloc(const float* dmsg_time, const float* dt, const int32_t* n_rows,
                                              int64_t max_rows, const float* time_w, const float* time_b,
                                              const mtgnn_dims* dims, float* d_time_w, float* d_time_b,
                                              hipStream_t stream);

/* Offline backward dependency scan and mixed-batch construction (Algorithm 1, Section IV-B), for
 * every worker p < n_workers and every synchronization window (Definition 1: `window` consecutive
 * batches of `batch` events; the last batch and window may be short).  For each (p, window) the
 * window's batches are scanned latest first: the batch's target events of p (source owned by p,
 * owner[src] == p) are kept and their remote destinations join the frontier F; then every event of
 * the batch whose source is remote and that touches F, visited latest first, becomes an auxiliary
 * replay event of p, and its remote endpoints join F.  Writes
 *   role      -- [n_workers, n_events] uint8: 0 = not in p's mixed batches, 1 = target of p,
 *                2 = auxiliary replay event of p;
 *   sync_bits -- [n_workers, n_windows, ceil(n_nodes / 32)] uint32: F at the end of each scan, the
 *                candidate boundary refresh set N_sync (bit n % 32 of word n / 32).
 * src, dst [n_events] int32 and owner [n_nodes] int32 (the node ownership map pi) are device arrays.
 * The result is the sequential algorithm's, bit for bit (no ordering freedom).  Errors: EINVAL. */
mtgnn_status mtgnn_dependency_scan(const int32_t* src, const int32_t* dst, int64_t n_events, const int32_t* owner,
                                   int64_t n_nodes, int32_t n_workers, int64_t batch, int32_t window, uint8_t* role,
                                   uint32_t* sync_bits, hipStream_t stream);

/* One worker's mixed batches (Eq. 5) from its roles: the events with role != 0 in stream order
 * (sort_t, as the stream is sorted by time), with the event-type mask.
 *   role      -- [n_events] uint8 (one worker's row of mtgnn_dependency_scan's output);
 *   eid_out   -- [n_events] int32 out: the event ids, batch after batch;
 *   flags_out -- [n_events] uint8 out: bit 0 set for auxiliary replay events (the mtgnn_batch flags);
 *   batch_off -- [ceil(n_events / batch) + 1] int32 out: batch s of the worker is entries
 *                batch_off[s] .. batch_off[s + 1] - 1; the last entry is the total.
 * Workspace: mtgnn_workspace_bytes(MTGNN_OP_MIXED_BATCHES, NULL, n_events, 0). */
mtgnn_status mtgnn_mixed_batches(const uint8_t* role, int64_t n_events, int64_t batch, int32_t* eid_out,
                                 uint8_t* flags_out, int32_t* batch_off, void* ws, size_t ws_bytes,
                                 hipStream_t stream);

/* ------------------------------------------------------------------ the JODIE variant
 * Section VII-A's second model.  Its memory phase uses mtgnn_aggregate_last and mtgnn_build_messages
 * as TGN's does; Update (Eq. 2) is a recurrent cell, and the embedding a projection of the memory in
 * time instead of the attention (no neighbour sampling).  The masked loss is mtgnn_link_loss with
 * d_attn = d_mem.  d_mem <= 256. */

/* JODIE's memory update (Eq. 2): for each aggregated row r < n_rows,
 *   h' = tanh(W_ih x + b_ih + W_hh h + b_hh),  x = msg[r], h = M[uniq[r]] (the first d_mem columns of
 *   msg[r]); memory[uniq[r]] = h' (rounded to the dtype), last_update[uniq[r]] = t of the winner.
 *   W_ih [d_mem, d_msg], W_hh [d_mem, d_mem] (dtype); b_ih, b_hh [d_mem] float32;
 *   save -- mtgnn_save_bytes(MTGNN_OP_RNN_UPDATE) bytes (h', float32) for the backward, or NULL.
 * Arguments and errors otherwise as mtgnn_gru_update. */
mtgnn_status mtgnn_rnn_update(const mtgnn_batch* b, const int32_t* uniq, const int32_t* winner,
                              const int32_t* n_rows, int64_t max_rows, const void* msg, const void* W_ih,
                              const void* W_hh, const float* b_ih, const float* b_hh, const mtgnn_dims* dims,
                              void* memory, float* last_update, void* save, void* ws, size_t ws_bytes,
                              hipStream_t stream);

/* Backward of mtgnn_rnn_update for d_mem = dL/dh' (the previous memory is detached): with
 * dpre = d_mem (1 - h'^2), dW_ih = dpre^T msg, dW_hh = dpre^T h, db_ih = db_hh = sum of dpre (overwritten),
 * and dmsg_time = dpre W_ih[:, 2 d_mem : 2 d_mem + d_time] (the message's time slice). */
mtgnn_status mtgnn_rnn_update_bwd(const float* d_mem, const void* save, const void* msg, const int32_t* n_rows,
                                  int64_t max_rows, const void* W_ih, const void* W_hh, const mtgnn_dims* dims,
                                  float* dW_ih, float* dW_hh, float* db_ih, float* db_hh, float* dmsg_time,
                                  void* ws, size_t ws_bytes, hipStream_t stream);

/* JODIE's time-projection embedding of each query q < n_q:
 *   z[q] = M[n] (1 + W_p Delta + b_p),  Delta = (q_t[q] - last_update[n]) * time_scale  (two float32
 *   operations), n = q_node[q], with the table after this step's update.
 *   W_p [d_mem] (the [d_mem, 1] weight), b_p [d_mem] float32; z [max_q, d_mem] float32 out. */
mtgnn_status mtgnn_time_projection(const int32_t* q_node, const float* q_t, const int32_t* n_q, int64_t max_q,
                                   const void* memory, const float* last_update, const float* W_p, const float* b_p,
                                   float time_scale, const mtgnn_dims* dims, float* z, hipStream_t stream);

/* Backward of mtgnn_time_projection for dz [max_q, d_mem]:
 *   dW_p, db_p [d_mem] (overwritten): the column sums over the queries of dz M Delta and dz M;
 *   d_mem [max_rows, d_mem] out, row r aligned with uniq[r]: the sum over the queries of node uniq[r]
 *     of dz (1 + W_p Delta + b_p), in query order (rows of uniq that no query names get 0; nodes not
 *     in uniq get nothing: the table is not differentiated across steps).
 * Deterministic (fixed-order sums).  Workspace: MTGNN_OP_TIME_PROJECTION_BWD with max_q. */
mtgnn_status mtgnn_time_projection_bwd(const int32_t* q_node, const float* q_t, const int32_t* n_q, int64_t max_q,
                                       const void* memory, const float* last_update, const float* W_p,
                                       const float* b_p, float time_scale, const float* dz, const int32_t* uniq,
                                       const int32_t* n_rows, int64_t max_rows, const mtgnn_dims* dims, float* dW_p,
                                       float* db_p, float* d_mem, void* ws, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------ adaptive runtime controller
 * The decisions of one worker's runtime controller (Section V, Algorithm 2), kept on the host:
 *   gradient-norm EMA (Eq. 6):   g_bar = g_r if g_bar was 0, else alpha g_r + (1 - alpha) g_bar;
 *   boundary decision (Eq. 7):   at a candidate refresh boundary r (r % interval == 0, Definition 1),
 *                                S_r = 0 (skip the refresh) iff r > 0, g_bar > 0 and g_{r-1} < tau_g g_bar;
 *   batch-time EMA (Eq. 8):      c_bar = c_r if c_bar was 0, else beta c_r + (1 - beta) c_bar;
 *   heavy load (Eq. 9):          H_r = 1 iff r > 0, c_bar > 0 and c_{r-1} > tau_c c_bar.
 * The paper fixes no values for alpha, beta, tau_g, tau_c; the caller chooses them. */
typedef struct {
  double alpha, beta;   /* EMA factors of the gradient norm and the batch time, in (0, 1] */
  double tau_g, tau_c;  /* thresholds, > 0 */
  int32_t interval;     /* K, the synchronization interval in batches, > 0 */
} mtgnn_controller_config;

typedef struct mtgnn_controller mtgnn_controller;   /* opaque, host memory */

/* Creates a controller in its initial state (every average and last value 0).  EINVAL on a NULL
 * argument or a value out of range.  Host-only; no HIP call. */
mtgnn_status mtgnn_controller_create(const mtgnn_controller_config* cfg, mtgnn_controller** out);
void mtgnn_controller_destroy(mtgnn_controller* c);
/* Before batch r: whether r is a candidate refresh boundary, the boundary decision S_r (0 when r is no
 * boundary) and the heavy-load mode H_r, from the state the previous observe left.  Any of the outputs
 * may be NULL. */
mtgnn_status mtgnn_controller_decide(const mtgnn_controller* c, int64_t r, int32_t* boundary, int32_t* sync,
                                     int32_t* heavy);
/* After batch r: its gradient norm g_r and batch time c_r (finite, >= 0; EINVAL otherwise) update the
 * averages and the last values. */
mtgnn_status mtgnn_controller_observe(mtgnn_controller* c, double grad_norm, double batch_time);
mtgnn_status mtgnn_controller_state(const mtgnn_controller* c, double* g_bar, double* g_last, double* c_bar,
                                    double* c_prev);

/* The gradient norm g_r of Eq. 6: sqrt of the sum of squares of every element of the n (<= 32) float32
 * tensors grads[i] (device pointers, host array) of sizes[i] (host array) elements, summed in double
 * precision in a fixed order (deterministic).  norm: a device double.  Workspace:
 * 8 * sum_i ceil(sizes[i] / 4096) bytes, rounded up to 256 (mtgnn_grad_norm_ws_bytes). */
size_t mtgnn_grad_norm_ws_bytes(const int64_t* sizes, int32_t n);
mtgnn_status mtgnn_grad_norm(const float* const* grads, const int64_t* sizes, int32_t n, double* norm, void* ws,
                             size_t ws_bytes, hipStream_t stream);

/* PruneAux (Eq. 10-11) of a mixed batch's event-type masks (mtgnn_batch flags, device, n entries): with
 * heavy != 0, every auxiliary replay event (bit 0: its source is not owned by the worker, the eligible
 * set of Eq. 10) gets bit 1 (pruned): the step then gives it no message, query or loss, as if removed;
 * target events are never touched.  With heavy == 0 bit 1 is cleared, restoring the mixed batch. */
mtgnn_status mtgnn_prune_aux(uint8_t* flags, int64_t n, int32_t heavy, hipStream_t stream);

/* Boundary cache refresh (Eq. 25): for every node n whose bit is set in sync_bits (bit n % 32 of word
 * n / 32, as mtgnn_dependency_scan writes the refresh set N_sync), memory row n and last_update[n] take
 * the authoritative table's values.  Other rows are not touched.  Tables: [n_nodes, d_mem] in the dims'
 * dtype and [n_nodes] float32, device. */
mtgnn_status mtgnn_cache_refresh(const uint32_t* sync_bits, int64_t n_nodes, const void* auth_memory,
                                 const float* auth_last_update, const mtgnn_dims* dims, void* memory,
                                 float* last_update, hipStream_t stream);

/* The parameter update of Algorithm 2: one Adam step (bias-corrected, step count t >= 1) over n (<= 32)
 * float32 parameter tensors in place, with their float32 moment buffers m, v; shadow (NULL, or per
 * tensor NULL or a bfloat16 buffer) receives the round-to-nearest-even bf16 copy of the updated
 * parameter (the storage weights of a bf16 run).  All tensor pointers are device pointers in host
 * arrays. */
typedef struct {
  double lr, beta1, beta2, eps;   /* the update's coefficients are formed in double, then used in float32 */
  int32_t t;
} mtgnn_adam_config;
mtgnn_status mtgnn_adam_step(float* const* params, const float* const* grads, float* const* m, float* const* v,
                             void* const* shadow, const int64_t* sizes, int32_t n, const mtgnn_adam_config* cfg,
                             hipStream_t stream);

/* Temporal adjacency of a whole stream (built once, offline; outside the step).
 * Event e = (src[e], dst[e], t[e]) with eid e gives two entries: (node src,
 * nbr dst, role 0) and (node dst, nbr src, role 1).  Entries are grouped by
 * node and sorted by (t, eid, role) within each node.
 * Precondition: the stream is sorted by (t, eid) ascending.
 *   csr_off [n_nodes+1] int64 out; csr_nbr, csr_eid int32 and csr_t float32 [2 n_events] out. */
mtgnn_status mtgnn_build_temporal_csr(const int32_t* src, const int32_t* dst, const float* t, int64_t n_events,
                                      int64_t n_nodes, int64_t* csr_off, int32_t* csr_nbr, float* csr_t,
                                      int32_t* csr_eid, void* ws, size_t ws_bytes, hipStream_t stream);

/* Launch timer (instrumentation for benchmarks; not part of the step).
 * mtgnn_timer_start arms it: each of the next `max_launches` launches whose
 * timer name equals `kernel` is bracketed by HIP events recorded on the
 * stream of that launch.  The names are the call-site names of the
 * matrix-product kernels ("gemm_kv_proj", "gemm_kv_dw", "gemm_kv_dx", "gemm")
 * and the function names of the other kernels (e.g. "k_attn_core").
 * mtgnn_timer_stop waits for the recorded events (host-blocking), returns
 * the summed duration in milliseconds and the number of timed launches, and
 * disarms the timer.  Host-side state: use from one host thread. */
mtgnn_status mtgnn_timer_start(const char* kernel, int max_launches);
mtgnn_status mtgnn_timer_stop(double* total_ms, int* launches);

/* Human-readable name of a status code (static storage). */
const char* mtgnn_status_string(int status);

/* The message of the last MTGNN_EHIP / validation failure on this host thread
 * ("" if none). */
const char* mtgnn_last_error(void);

/* ABI version (major * 100 + minor). */
int mtgnn_version(void);

#ifdef __cplusplus
}
#endif

#endif /* MTGNN_H */

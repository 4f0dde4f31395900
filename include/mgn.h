/*
 * libmgn -- one MeshGraphNets training step (forward and backward) on one
 * GPU's mesh partition, for AMD MI355X (gfx950).
 *
 * The network is the encode-process-decode model of the paper (section
 * "Model"; Algorithm 1 "Training of distributed MeshGraphNets"): EncNode and
 * EncEdge map node and edge features to latent size l, K message-passing
 * blocks update edge and node latents, DecNode maps node latents to outputs.
 * Readings where the paper is silent:
 *   - every MLP has `depth` Linear layers of width l with ReLU between them
 *     and, except the decoder, ends in an affine LayerNorm (biased variance,
 *     epsilon ln_eps);
 *   - block k, edge e = (s -> r):  m_e = LN(MLP([e_e | v_s | v_r])),
 *     e_e <- e_e + m_e;  agg_r = sum of m_e over the edges into r;
 *     v_r <- v_r + LN(MLP([v_r | agg_r]));
 *   - the partition holds the edges whose receiver it owns (section
 *     "Methodology": halo of depth one); halo node latents at the input of
 *     block k come in as halo[k]; the caller exchanges them between the
 *     stages of a staged step (mgn_forward_block, mgn_copy_latents and
 *     mgn_add_latent_grads below) or supplies them all up front.
 *
 * Conventions
 *   - Every function returns an mgn_status; MGN_OK is 0.  On error nothing is
 *     enqueued and no state changes; mgn_last_error() explains.
 *   - Device pointers are caller-owned device memory (any allocator).  Host
 *     pointers are plain host memory.  The library owns only the parameters
 *     (fp32 master copy plus packed copies for the kernels).
 *   - Work is enqueued asynchronously on the given HIP stream (a hipStream_t
 *     passed as void*; NULL is the default stream).  Only mgn_set_params,
 *     mgn_get_params (host side) and mgn_graph_validate synchronise.
 *   - Sums are taken in a fixed order without atomics: results are bitwise
 *     reproducible for the same inputs.
 *   - Indices are int32; element offsets are 64-bit internally.
 */
#ifndef LIBMGN_MGN_H
#define LIBMGN_MGN_H
#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MGN_OK = 0,
  MGN_E_ARG = 1,          /* bad argument: null/misaligned pointer, bad size */
  MGN_E_GRAPH = 2,        /* graph arrays fail validation */
  MGN_E_STATE = 3,        /* call out of order (e.g. backward before forward) */
  MGN_E_NOMEM = 4,        /* device allocation failed, or workspace too small */
  MGN_E_HIP = 5,          /* a HIP runtime call or kernel launch failed */
  MGN_E_UNSUPPORTED = 6   /* configuration outside what the kernels handle */
} mgn_status;

typedef enum {
  MGN_FP32 = 0,  /* fp32 storage, fp32 MFMA (v_mfma_f32_16x16x4_f32) */
  MGN_BF16 = 1   /* bf16 MFMA inputs and bf16 edge-latent stream; fp32
                    accumulation, LayerNorm, residual of node latents and
                    every receiver / sender sum (mixed precision, cf. the
                    paper's section "Performance Study") */
} mgn_precision;

typedef struct {
  int32_t latent;    /* l: 64, 128 or 256 */
  int32_t n_blocks;  /* K >= 0 message-passing blocks */
  int32_t depth;     /* Linear layers per MLP: 2 or 3 */
  int32_t node_in;   /* node features: 1..32 (11 = 3 coords + 5 flow + 3 type) */
  int32_t edge_in;   /* edge features: 1..32 (4 = displacement + norm) */
  int32_t node_out;  /* outputs per node: 1..16 (5) */
  int32_t precision; /* mgn_precision */
  float ln_eps;      /* LayerNorm epsilon, > 0 (1e-5) */
} mgn_config;

typedef struct mgn_model mgn_model;
typedef void* mgn_stream;

/* Partition-local graph (device arrays, caller-owned, int32):
 *   row_ptr [n_owned + 1]  receiver CSR: local edges of owned receiver r are
 *                          row_ptr[r] .. row_ptr[r+1]-1;
 *   send    [n_edges]      local id of each local edge's sender
 *                          (0..n_owned-1 owned, n_owned.. halo);
 *   trow_ptr[n_owned + n_halo + 1], tedge[n_edges]  transposed CSR: the local
 *                          edges sent by node n, ascending.
 * mgn_graph_build produces these arrays on the host. */
typedef struct {
  int64_t n_owned, n_halo, n_edges;
  const int32_t* row_ptr;
  const int32_t* send;
  const int32_t* trow_ptr;
  const int32_t* tedge;
} mgn_graph;

/* Creates a model for `cfg` (host state only; the parameters' device memory
 * is allocated on the current HIP device by the first mgn_set_params).
 * Errors: MGN_E_ARG (null), MGN_E_UNSUPPORTED (latent/depth/dims out of
 * range). */
mgn_status mgn_create(const mgn_config* cfg, mgn_model** out);
/* Frees the model's device memory; NULL is allowed. */
void mgn_destroy(mgn_model* m);
/* Message for the last failed call on `m`, or for the last failed call of
 * this thread without a model when m is NULL.  Never NULL. */
const char* mgn_last_error(const mgn_model* m);

/* Number of fp32 parameters.  Flat layout, in this order: EncNode, EncEdge,
 * then for k = 0..K-1 the edge MLP and the node MLP of block k, then DecNode.
 * Per MLP: for each Linear W[out][in] row-major then b[out]; then LayerNorm
 * gamma[l], beta[l] (not for DecNode).  Edge Linear-1 input columns are
 * [e | v_sender | v_receiver], node Linear-1 input columns are [v | agg]. */
int64_t mgn_param_count(const mgn_model* m);

/* Copies parameters in (src: host or device fp32 [param_count]) and refreshes
 * the packed copies the kernels use.  Synchronises `stream`.  MGN_E_NOMEM if
 * the first call cannot allocate the model's device memory. */
mgn_status mgn_set_params(mgn_model* m, const float* src, int src_on_device, mgn_stream stream);
/* Algorithm 1's update after the (accumulated) gradient: theta <- theta -
 * lr * grad for every parameter (one fused multiply-add each), then the
 * packed copies are refreshed.  grad: device fp32 [param_count] (e.g. the
 * d_params of mgn_backward).  Enqueued on `stream`, no synchronisation; a
 * step in progress is dropped (its backward would no longer match the
 * parameters).  MGN_E_ARG for a NULL grad or a non-finite lr, MGN_E_STATE
 * before mgn_set_params. */
mgn_status mgn_sgd_step(mgn_model* m, const float* grad, float lr, mgn_stream stream);
/* Copies the fp32 parameters out (host or device).  Synchronises `stream`. */
mgn_status mgn_get_params(const mgn_model* m, float* dst, int dst_on_device, mgn_stream stream);

/* ---- host-side graph preprocessing (section "Methodology": partition plus
 * depth-1 halo; Algorithm 1's send/receive masks, built once per mesh) ---- */

/* Slab partition standing in for METIS: nodes ranked by (key, node id); the
 * node of rank q goes to part floor(nparts * q / n).  Host arrays. */
mgn_status mgn_partition_slabs(const int32_t* key, int64_t n, int32_t nparts, int32_t* part);
/* Sizes of part p's local graph from the global directed edge list (host):
 * sizes[0] owned nodes, sizes[1] halo nodes (senders of owned-receiver edges
 * outside p), sizes[2] local edges (receiver in p). */
mgn_status mgn_graph_sizes(const int32_t* send, const int32_t* recv, int64_t n_edges, const int32_t* part,
                           int64_t n_nodes, int32_t p, int64_t* sizes);
/* Builds part p's local graph into caller-allocated host arrays: local ids
 * are the owned nodes by ascending global id, then the halo nodes by
 * ascending global id; local edges sorted by (receiver, sender, global edge
 * id).  row_ptr[n_owned+1], send_local[E], eperm[E] (global id of each local
 * edge), trow_ptr[n_owned+n_halo+1], tedge[E], l2g[n_owned+n_halo]. */
mgn_status mgn_graph_build(const int32_t* send, const int32_t* recv, int64_t n_edges, const int32_t* part,
                           int64_t n_nodes, int32_t p, int32_t* row_ptr, int32_t* send_local, int32_t* eperm,
                           int32_t* trow_ptr, int32_t* tedge, int32_t* l2g);
/* Checks a device graph (copies it to the host; synchronises `stream`) and
 * records it as the graph mgn_forward may run on.  MGN_E_GRAPH names the
 * first violated property. */
mgn_status mgn_graph_validate(mgn_model* m, const mgn_graph* g, mgn_stream stream);

/* ---- the training step ---- */

/* Edge-stream checkpointing (bf16 precision only).  interval 0 (the
 * default) keeps every block's inputs for the backward pass.  interval s >= 1
 * keeps the edge latents of blocks 0, s, 2s, ... only, and of the node stream
 * only the bf16 copy: the backward pass recomputes each block's edge latents
 * from the nearest checkpoint at or below it and the block's aggregate by
 * one more edge forward, and runs the edge backward in receiver chunks of
 * about chunk_edges edges (0: 8Mi).  Same computation (the weight-gradient
 * sums over chunks add in another order); the workspace then holds
 * ceil(K/s) + 1 edge-latent copies instead of K.  Takes effect for the next
 * mgn_workspace_size / mgn_forward (a pending backward is dropped).
 * MGN_E_UNSUPPORTED for fp32 models, MGN_E_ARG for negative arguments. */
mgn_status mgn_set_recompute(mgn_model* m, int32_t interval, int64_t chunk_edges);

/* First-Linear stash of the row-split edge kernels (bf16, latent 64, or
 * latent 128 at MLP depth 2; section "Model", the edge MLP of each block).
 * Without checkpointing, the backward pass recomputes each block's
 * first-Linear ReLU output h_1 from e^k and the kept node projections, and
 * writes it for the layer-2 weight gradient.  n_blocks > 0 makes the forward
 * keep h_1 of the last min(n_blocks, K) blocks (E x latent bf16 each, in the
 * workspace); their backward reads it instead of e^k and the projections
 * and writes nothing in its place, so their forwards share one projection
 * slot (n_nodes x 2 latent fp32) instead of keeping one each.  Identical results (h_1 is the same
 * bf16 value either way); less traffic for more workspace.  Ignored by
 * other kernels (the streaming kernels keep every block's h_1 anyway),
 * with checkpointing and in inference.  Takes effect for the next
 * mgn_workspace_size / mgn_forward (a pending step is dropped).
 * MGN_E_ARG for a negative count. */
mgn_status mgn_set_h1_stash(mgn_model* m, int32_t n_blocks);

/* Forward-only plan (inference on a whole mesh, the paper's section
 * "Results": a single GPU holds a complete stator domain for inference).
 * on != 0: the workspace holds one working copy of each stream (node
 * latents and their bf16 copy in a ping-pong pair, the edge latents updated
 * in place) and no backward buffers; mgn_backward then returns MGN_E_STATE.
 * Same arithmetic as the training plan: outputs are bitwise equal.  While on,
 * the edge-stream checkpointing setting (mgn_set_recompute) is ignored.
 * Takes effect for the next mgn_workspace_size / mgn_forward (a pending step
 * is dropped). */
mgn_status mgn_set_inference(mgn_model* m, int32_t on);

/* Next-step rollout (section "Model": the network predicts the increment,
 * q_{t+1} = p + q_t): node_feat[i][col0 + j] += out[i][j] for i < n,
 * j < node_out (device fp32; row strides node_in and node_out).  With the
 * default features (3 coordinates, 5 flow quantities, 3 type flags) col0 = 3.
 * MGN_E_ARG unless col0 + node_out <= node_in. */
mgn_status mgn_rollout_update(const float* out, int64_t n, int32_t node_out, float* node_feat, int32_t node_in,
                              int32_t col0, mgn_stream stream);

/* Normalize (Algorithm 1: the increments, node features and edge features
 * are normalised before the encoders), read as an online standardisation
 * per feature column.  stats is a device array of 1 + 2 cols doubles,
 * [n, column sums, column sums of squares] over every row accumulated so
 * far (all zero for a fresh normaliser; the caller owns it, one per kind of
 * input).  mgn_norm_accumulate adds the rows of x [rows][cols] (device fp32)
 * to it, summing in fp64 in a fixed order (no atomics: the same inputs give
 * the same bits); work is a device scratch array of at least
 * MGN_NORM_WORK_PER_COL * cols doubles, overwritten.  mgn_norm_apply writes
 * out[i][c] = (x[i][c] - mean_c) / max(std_c, eps) rounded from fp64 once,
 * with mean_c = sum / n and std_c the population deviation (no rows
 * accumulated: the identity); out may equal x.  Both are asynchronous on
 * `stream`.  MGN_E_ARG for rows < 0, cols outside 1 .. MGN_NORM_MAX_COLS,
 * eps <= 0, or a NULL / misaligned pointer (8-byte stats and work, 4-byte
 * x and out). */
#define MGN_NORM_MAX_COLS 64
#define MGN_NORM_WORK_PER_COL 1024
mgn_status mgn_norm_accumulate(const float* x, int64_t rows, int32_t cols, double* stats, double* work,
                               mgn_stream stream);
mgn_status mgn_norm_apply(const float* x, int64_t rows, int32_t cols, const double* stats, double eps, float* out,
                          mgn_stream stream);

/* Device workspace mgn_forward/mgn_backward need for graph g (bytes) under
 * the model's checkpointing setting. */
mgn_status mgn_workspace_size(const mgn_model* m, const mgn_graph* g, size_t* bytes);

/* Forward pass of one partition: Algorithm 1's forward (EncNode, EncEdge,
 * the K GraphNetBlocks with the halo latents of block k read from halo[k],
 * DecNode; section "Model": encoder, processor, decoder).  Device pointers:
 *   node_feat [n_owned][node_in], edge_feat [n_edges][edge_in] in local edge
 *   order, halo [K][n_halo][latent] (NULL iff n_halo == 0 or K == 0; 16-byte
 *   aligned), out [n_owned][node_out], workspace (256-byte aligned, at least
 *   mgn_workspace_size bytes; caller-owned).
 * g must be the graph last passed to mgn_graph_validate.  The pointers and
 * their contents must stay valid and unchanged until mgn_backward.
 * MGN_E_STATE without parameters or a validated graph, MGN_E_NOMEM when
 * ws_bytes is too small, MGN_E_ARG for NULL or misaligned pointers. */
mgn_status mgn_forward(mgn_model* m, const mgn_graph* g, const float* node_feat, const float* edge_feat,
                       const float* halo, float* out, void* workspace, size_t ws_bytes, mgn_stream stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops, harnesses that forbid hipMalloc): mgn_forward with
 * its workspace in a library-owned static device array of
 * MGN_NOALLOC_WS_MAX bytes, one per GPU, held until the process ends.  Same
 * arguments as mgn_forward without workspace / ws_bytes; same launches and
 * results.  Allocates nothing (no hipMalloc, no events).  Errors:
 * MGN_E_NOMEM when mgn_workspace_size for (m, g) exceeds
 * MGN_NOALLOC_WS_MAX (nothing is enqueued); MGN_E_STATE when launch timing
 * is on; otherwise as mgn_forward.  Every call on one GPU uses that GPU's one
 * array, which keeps the last call's contents: calls (from any model) that
 * overlap on one GPU race, and a later mgn_backward of this forward is valid
 * only while no other call has used the array since. */
#define MGN_NOALLOC_WS_MAX (128u << 20)
mgn_status mgn_forward_noalloc(mgn_model* m, const mgn_graph* g, const float* node_feat, const float* edge_feat,
                               const float* halo, float* out, mgn_stream stream);

/* Backward pass of the last forward (Algorithm 1: Backprop of the loss
 * through DecNode, the K blocks in reverse and the encoders; section
 * "Methodology": the halo gradients are what the owners receive).
 * d_out [n_owned][node_out] = dL/dout.
 * d_params [param_count] receives dL/dtheta (overwritten, or added to when
 * accumulate != 0: gradient accumulation of Algorithm 1).  d_halo
 * [K][n_halo][latent] (NULL allowed; 16-byte aligned) receives dL/dhalo,
 * overwritten: the gradients the halo owners would receive (section
 * "Methodology": backward gradient exchange).
 * Several backward calls may follow one forward.  With edge-stream
 * checkpointing (mgn_set_recompute) the first of them reads the last
 * block's aggregate where the forward left it and later ones recompute it;
 * a backward captured into a HIP graph records the choice made at capture,
 * so each replay of such a graph must follow a replay of the forward. */
mgn_status mgn_backward(mgn_model* m, const float* d_out, float* d_params, int accumulate, float* d_halo,
                        mgn_stream stream);

/* ---- the step in stages, for several partitions stepped in lockstep ----
 *
 * Algorithm 1 exchanges the halo after every message-passing block: halo
 * node latents forward (owners -> partitions holding them as halo), and in
 * the backward the halo gradients back to the owners (section
 * "Methodology": forward halo exchange and backward gradient exchange).
 * mgn_forward is exactly
 *     mgn_forward_begin; mgn_forward_block x K; mgn_forward_end
 * and mgn_backward is
 *     mgn_backward_begin; mgn_backward_block x K; mgn_backward_end,
 * so a caller stepping P partitions of one mesh (one model each, same
 * parameters) can exchange between the stages:
 *   forward:  begin (all parts); for k = 0..K-1: for every (part p, owner q):
 *             mgn_copy_latents(q -> p's halo[k]); mgn_forward_block (all parts);
 *             end (all parts);
 *   backward: begin (all); for k = K-1..0: mgn_backward_block (all); for every
 *             (p, q): mgn_add_latent_grads(p's d_halo[k] -> q); end (all).
 * With d_params shared and accumulate = 1 for every part but the first, the
 * parts' gradients add up to the gradient of the unpartitioned network.
 * Every stage enqueues on the given stream; a stage called out of order
 * returns MGN_E_STATE and enqueues nothing.  Errors inside a stage leave the
 * step unusable (start again with mgn_forward_begin). */

/* Arguments, checks and ownership as mgn_forward; runs the encoders.  halo
 * may be filled block by block: halo[k] is read when block k runs. */
mgn_status mgn_forward_begin(mgn_model* m, const mgn_graph* g, const float* node_feat, const float* edge_feat,
                             const float* halo, float* out, void* workspace, size_t ws_bytes, mgn_stream stream);
/* Runs the next message-passing block (k = 0, 1, ..., K-1 in turn). */
mgn_status mgn_forward_block(mgn_model* m, mgn_stream stream);
/* Runs the decoder after the K blocks; the step is then ready for a backward. */
mgn_status mgn_forward_end(mgn_model* m, mgn_stream stream);
/* Arguments and checks as mgn_backward; runs the decoder's backward. */
mgn_status mgn_backward_begin(mgn_model* m, const float* d_out, float* d_params, int accumulate, float* d_halo,
                              mgn_stream stream);
/* Runs the backward of the next block (k = K-1, ..., 0 in turn): writes
 * d_halo[k] and leaves dL/dv^k (owned node latents at block k's input). */
mgn_status mgn_backward_block(mgn_model* m, mgn_stream stream);
/* Runs the encoders' backward after the K blocks. */
mgn_status mgn_backward_end(mgn_model* m, mgn_stream stream);

/* Exchange lists between part p and its neighbour q (host arrays; Algorithm
 * 1's create_masks, built once per mesh): the halo nodes of p that q owns,
 * in ascending halo index.  recv_idx[i] = halo index j of such a node in p
 * (p's local id n_owned_p + j), send_rows[i] = its local id in q.  Inputs:
 * l2g_p [n_owned_p + n_halo_p] and l2g_q [n_owned_q + ...] from
 * mgn_graph_build, part [n_nodes].  recv_idx, send_rows: caller arrays of
 * n_halo_p entries; *count receives the number written.  MGN_E_GRAPH if q's
 * owned list is not ascending global ids of part q or misses a node. */
mgn_status mgn_halo_masks(const int32_t* l2g_p, int64_t n_owned_p, int64_t n_halo_p, const int32_t* part,
                          int64_t n_nodes, const int32_t* l2g_q, int64_t n_owned_q, int32_t q, int32_t* recv_idx,
                          int32_t* send_rows, int64_t* count);
/* Forward exchange (device arrays): halo_k[recv_idx[i]][:] = v[send_rows[i]][:]
 * for i < n, where v are the owner's node latents at the input of its next
 * block (after mgn_forward_begin: v^0; after block k-1: v^k; after the
 * forward: v^K).  halo_k is a [n_halo][latent] fp32 block of the receiving
 * part's halo buffer (16-byte aligned).  Pairs with an index outside
 * [0, owner's n_owned) or [0, n_halo) are skipped.  Enqueued on `stream`. */
mgn_status mgn_copy_latents(const mgn_model* owner, const int32_t* send_rows, const int32_t* recv_idx, int64_t n,
                            float* halo_k, int64_t n_halo, mgn_stream stream);
/* Backward exchange (device arrays): dv[send_rows[i]][:] += d_halo_k[recv_idx[i]][:]
 * for i < n, where dv is the owner's dL/dv of its last backward stage
 * (after mgn_backward_block for block k: dL/dv^k) and d_halo_k the
 * [n_halo][latent] block k of the holding part's d_halo.  send_rows must be
 * distinct within one call (lists from mgn_halo_masks are); calls adding
 * into one owner run in stream order, so the sum has a fixed order.
 * Out-of-range pairs are skipped, as above. */
mgn_status mgn_add_latent_grads(mgn_model* owner, const float* d_halo_k, int64_t n_halo, const int32_t* recv_idx,
                                const int32_t* send_rows, int64_t n, mgn_stream stream);

/* One exchange list of a lockstep step (device index arrays, n entries, from
 * mgn_halo_masks): the halo rows recv_idx of part `part` are the node rows
 * send_rows of part `owner`. */
typedef struct {
  int32_t part, owner;
  const int32_t* recv_idx;
  const int32_t* send_rows;
  int64_t n;
} mgn_halo_link;

/* The staged forward of n_parts parts (one model each, same configuration
 * and parameters) in Algorithm 1's order: every part's encoders; for each
 * block, every link's mgn_copy_latents into halo[part] (block k of a
 * [K][n_halo][latent] buffer), then every part's block; every part's
 * decoder.  Per part p: graphs[p], node_feat[p], edge_feat[p], halo[p]
 * (NULL for a part without halo), out[p], workspace[p], ws_bytes[p] as for
 * mgn_forward.  Links are applied in array order.  Errors as the calls it
 * makes (on an error the parts' steps are dropped). */
mgn_status mgn_lockstep_forward(int32_t n_parts, mgn_model* const* models, const mgn_graph* graphs,
                                const float* const* node_feat, const float* const* edge_feat, float* const* halo,
                                float* const* out, void* const* workspace, const size_t* ws_bytes,
                                const mgn_halo_link* links, int32_t n_links, mgn_stream stream);
/* The staged backward of the same parts: every part's decoder backward;
 * for k = K-1 .. 0 every part's block backward, then every link's
 * mgn_add_latent_grads from d_halo[part]; every part's encoder backward.
 * d_params (device [param_count]) receives the sum of the parts' gradients
 * in part order (overwritten by the first part unless accumulate != 0);
 * d_halo[p] [K][n_halo][latent] is part p's halo-gradient buffer. */
mgn_status mgn_lockstep_backward(int32_t n_parts, mgn_model* const* models, const float* const* d_out,
                                 float* d_params, int accumulate, float* const* d_halo, const mgn_halo_link* links,
                                 int32_t n_links, mgn_stream stream);

/* Masked mean squared error (Algorithm 1: local squared error, mean over the
 * loss-masked nodes and outputs) and its gradient, device pointers:
 * out, target [n][d]; mask [n] (NULL = all rows); loss [2]: loss[0] = loss,
 * loss[1] = 2/(rows*d) (scratch); d_out [n][d] (also holds per-workgroup
 * partial sums before the gradient overwrites it). */
mgn_status mgn_mse_grad(const float* out, const float* target, const uint8_t* mask, int64_t n, int32_t d,
                        float* loss, float* d_out, mgn_stream stream);

/* The global mean of Algorithm 1 over several parts (its loss all-reduce):
 * as mgn_mse_grad for one part's rows, but the mean runs over global_rows
 * loss-masked rows of all parts together (>= 1; the host knows it from the
 * masks).  loss[0] = this part's share, sum of its squared errors /
 * (global_rows * d); the parts' shares add up to the global loss.  d_out =
 * 2 (out - target) / (global_rows * d) on masked rows, 0 elsewhere: the
 * gradient of the global loss. */
mgn_status mgn_mse_grad_global(const float* out, const float* target, const uint8_t* mask, int64_t n, int32_t d,
                               int64_t global_rows, float* loss, float* d_out, mgn_stream stream);

/* ---- kernel timing (measurement; the paper's section "Performance Study"
 * times its step with host-synchronised streams, this records HIP events on
 * the stream around each launch instead) ---- */
typedef enum {
  MGN_T_ENCODE = 0,        /* EncNode, EncEdge forward */
  MGN_T_EDGE_FWD = 1,      /* fused edge half of a block, forward */
  MGN_T_NODE_FWD = 2,      /* fused node half of a block, forward */
  MGN_T_DECODE = 3,        /* DecNode forward */
  MGN_T_EDGE_BWD = 4,      /* fused edge half, backward with recompute */
  MGN_T_NODE_BWD = 5,      /* node half, decoder and encoders, backward */
  MGN_T_INPUT_GRAD = 6,    /* node gradients through the edge MLP's first Linear */
  MGN_T_WEIGHT_GRAD = 7,   /* weight-gradient GEMMs and fixed-order reductions */
  MGN_T_OTHER = 8,         /* planning, loss */
  MGN_T_NODE_PROJ = 9,     /* per-node products of the edge MLP's first Linear (row-split edge kernels) */
  MGN_T_EXCHANGE = 10,     /* halo exchange between partitions (mgn_copy_latents, mgn_add_latent_grads),
                              timed on the owner's model */
  MGN_T_COUNT = 11
} mgn_timer;
/* Starts (enable != 0) or stops recording; starting clears earlier records. */
mgn_status mgn_timing_enable(mgn_model* m, int enable);
/* Sum of the recorded launch durations of one timer class (milliseconds) and
 * the number of launches.  Waits for the recorded events. */
mgn_status mgn_timing_read(mgn_model* m, int timer, double* ms_total, int64_t* launches);

#ifdef __cplusplus
}
#endif
#endif

/*
 * CPU oracle for the MeshGraphNets training step -- TEST INFRASTRUCTURE.
 *
 * A plain, slow, float64 implementation of what the GPU library computes, used
 * only by the tests, the smoke check and the CPU-baseline leg of the benchmark
 * to check the GPU results.  It shares no code, header, table or helper with
 * the GPU library.
 *
 * Model (paper, section "Model" and Algorithm 1 "Training of distributed
 * MeshGraphNets"): node and edge encoders, K message-passing blocks, a node
 * decoder.  Where the paper is silent the readings are:
 *   - every MLP has `depth` Linear layers of width `latent` with ReLU between
 *     them; every MLP except the decoder ends in an affine LayerNorm
 *     (biased variance, epsilon ln_eps);
 *   - edge block:  m_e = LN(MLP([e_e | v_s | v_r])),  e_e <- e_e + m_e,
 *     agg_r = sum of m_e over edges into r;
 *     node block:  v_r <- v_r + LN(MLP([v_r | agg_r]))  for owned r;
 *   - halo latents: v_h at the input of block k is halo[k][h] (the depth-1
 *     halo of section "Methodology"; exchange between blocks, Algorithm 1);
 *   - a partition holds exactly the edges whose receiver it owns.
 * All arithmetic is float64; sums run in ascending index order.
 */
#ifndef MGN_ORACLE_H
#define MGN_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* bf16 != 0 selects the mixed-precision reading of the paper's automatic
 * mixed precision (section "Performance Study"): every Linear's input
 * activations and weights, and every backward gradient that feeds a matrix
 * product, are rounded to bfloat16 (as binary32 values, then to nearest
 * with 8 significant bits, ties to even) before the
 * product; the edge-latent stream is stored rounded, and so is its gradient
 * dL/de^k (the sum of the residual's and the MLP input's contributions,
 * rounded once per block, as the gradient of a bfloat16 tensor is itself
 * bfloat16); biases, LayerNorm, the node-latent stream and its gradient,
 * every other sum and every bias / LayerNorm gradient stay in full
 * precision.  bf16 == 0: float64 throughout. */
typedef struct {
  int32_t latent, n_blocks, depth, node_in, edge_in, node_out;
  double ln_eps;
  int32_t bf16;
} orc_cfg;

/* Number of parameters in the flat layout: EncNode, EncEdge, per block
 * {edge MLP, node MLP}, DecNode; per Linear W[out][in] then b[out]; per
 * LayerNorm gamma then beta. */
int64_t orc_param_count(const orc_cfg* c);

/* Slab partition used in place of METIS: nodes ranked by (key, id); node of
 * rank q goes to part floor(nparts*q/n).  Returns 0, or -1 on bad arguments. */
int orc_partition(const int32_t* key, int64_t n, int32_t nparts, int32_t* part);

/* Partition-local graph of part p (section "Methodology": depth-1 halo).
 * sizes[0..2] = owned nodes, halo nodes, local edges. */
int orc_graph_sizes(const int32_t* send, const int32_t* recv, int64_t n_edges,
                    const int32_t* part, int64_t n_nodes, int32_t p, int64_t* sizes);
/* Local ids: owned nodes by ascending global id, then halo nodes by ascending
 * global id.  Local edges (receiver owned) sorted by (receiver, sender, global
 * edge id): row_ptr[n_owned+1], send_local[E], eperm[E] (global edge id).
 * Transposed CSR: trow_ptr[n_owned+n_halo+1], tedge[E] (local edge ids grouped
 * by sender, ascending).  l2g[n_owned+n_halo]. */
int orc_graph_build(const int32_t* send, const int32_t* recv, int64_t n_edges,
                    const int32_t* part, int64_t n_nodes, int32_t p,
                    int32_t* row_ptr, int32_t* send_local, int32_t* eperm,
                    int32_t* trow_ptr, int32_t* tedge, int32_t* l2g);

/* Edge features of section "Model": (x_s - x_r)/h and |x_s - x_r|/h. */
int orc_edge_features(const double* coords, const int32_t* send, const int32_t* recv,
                      int64_t n_edges, double h, double* out);

/* Receiver-CSR sum: agg[r] = sum over local edges e of r (ascending e) of m[e]. */
int orc_scatter_sum(int64_t n_owned, const int32_t* row_ptr, const double* m, int32_t width,
                    double* agg);

/* Forward (and, when d_out != NULL, backward) of one training step on one
 * partition-local graph.  out[n_owned][node_out]; d_params[param_count]
 * (overwritten); d_halo[K][n_halo][latent] (overwritten, may be NULL);
 * v_all[(K+1)][n_owned+n_halo][latent] and e_all[(K+1)][n_edges][latent]
 * receive every block's node and edge latents when non-NULL (halo rows of the
 * last block are zero).  Returns 0, or -1 on bad arguments. */
int orc_step(const orc_cfg* c, int64_t n_owned, int64_t n_halo, int64_t n_edges,
             const int32_t* row_ptr, const int32_t* send, const double* params,
             const double* node_feat, const double* edge_feat, const double* halo,
             const double* d_out, double* out, double* d_params, double* d_halo,
             double* v_all, double* e_all);

/* Masked mean squared error over n rows of d outputs (Algorithm 1: local sum of
 * squared errors, mean over the loss-masked nodes); d_out = dL/dout. */
int orc_mse_grad(const double* out, const double* target, const uint8_t* mask, int64_t n,
                 int32_t d, double* loss, double* d_out);

/* One part's share of the global masked mean over global_rows rows of all
 * parts (0: this part's own masked rows); d_out = gradient of the global loss. */
int orc_mse_grad_global(const double* out, const double* target, const uint8_t* mask, int64_t n,
                        int32_t d, int64_t global_rows, double* loss, double* d_out);

/* Algorithm 1's update with learning rate eta: params -= lr * grad (n entries). */
int orc_sgd_step(double* params, const double* grad, int64_t n, double lr);

/* Next-step rollout: node_feat[i][col0 + j] += out[i][j] (q_{t+1} = p + q_t). */
int orc_rollout_update(double* node_feat, int64_t n, int32_t node_in, const double* out, int32_t node_out,
                       int32_t col0);

/* Normalize (Algorithm 1): online per-column standardisation.  stats holds
 * 1 + 2 cols doubles [n, column sums, column sums of squares], zero for a
 * fresh normaliser; accumulate adds rows to it, apply writes
 * (x - mean) / max(std, eps).  Return -1 on bad arguments. */
int orc_norm_accumulate(const double* x, int64_t rows, int32_t cols, double* stats);
int orc_norm_apply(const double* x, int64_t rows, int32_t cols, const double* stats, double eps, double* out);

#ifdef __cplusplus
}
#endif
#endif

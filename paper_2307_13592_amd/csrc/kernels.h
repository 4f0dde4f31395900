// Host-visible launch interface of the libmgn kernels (internal; the public
// C ABI is include/mgn.h).  Every launcher enqueues asynchronously on the
// given stream and returns the hipError_t of the launch.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "device_common.h"

namespace mgn {

enum Prec { F32 = 0, BF16 = 1 };
enum RowKind { ENC_NODE = 0, ENC_EDGE = 1, NODE_BLOCK = 2, DECODER = 3 };

// ---------------------------------------------------------------- args ---
struct RowsFwdArgs {
  Mlp mlp;
  int64_t rows;
  int fin, fout;
  const float* in0;  // ENC: features [rows][fin]; NODE/DEC: v [rows][L]
  const float* in1;  // NODE: aggregated messages [rows][L]
  void* out;         // ENC_NODE, NODE, DEC: fp32; ENC_EDGE: storage type
  void* out16;       // ENC_NODE, NODE in bf16 mode: bf16 copy of the output rows (or null)
  const void* in0_16;  // NODE, bf16 T-form kernel: bf16 copy of v (the product operand), or null
  void* hid_out;       // NODE, bf16 T-form kernel: first Linear's ReLU output [rows][L] bf16, or null
  float eps;
};

struct EdgeFwdArgs {
  Mlp mlp;
  const int32_t* row_ptr;
  const int32_t* send;
  const int32_t* erecv;
  const int32_t* unit_r;
  const int32_t* n_units;
  const float* V;  // block input, owned rows [n_owned][L]
  const float* H;  // block input, halo rows [n_halo][L]
  const void* V16;  // bf16 mode: bf16 copy of the block input, owned then halo rows [n_owned+n_halo][L]
  int64_t n_owned;
  const void* Ein;  // edge latents in [E][L] (storage type)
  void* Eout;       // edge latents out, or null (last block)
  float* agg;       // [n_owned][L]
  const float* proj;  // node projections [n_local][2L] (row-split kernels), else unused
  void* hid_out;      // streaming and row-split kernels: the first Linear's ReLU output [E][L] (storage type) kept for the
                      // backward, or null
  float eps;
};

struct RowsBwdArgs {
  Mlp mlp;
  int64_t rows;
  int fin, fout;
  const float* in0;
  const float* in1;
  const void* in0_16;  // NODE / DEC: bf16 rows [rows][L] read instead of in0 when set
  const void* hid_in;  // NODE, bf16 T-form kernel: the forward's first-Linear ReLU output [rows][L]
  const float* dm;   // gradient w.r.t. the MLP output (LN output; dOut for the decoder)
  const uint16_t* dm16;  // ENC_EDGE in bf16 mode: that gradient as bf16 rows [rows][L] (dL/de^0), read instead of dm
  float* dx0;        // NODE: dv^k owned part (= dm + dX_v); DEC: dv^K
  float* dx1;        // NODE: d agg
  void* delta[3];    // storage type [rows][L]: gradient at each Linear's output
  void* hid[2];      // storage type [rows][L]: inputs of Linear 1 .. D-1
  float* vpart;      // [grid][nvec] per-workgroup bias / LayerNorm gradients
  int nvec;
  float eps;
  float* w1_part;    // ENC_EDGE, T-form kernel: when set, per-wave partials [waves][L][fin] of the
                     // first Linear's weight gradient instead of storing delta[0] (rows_rt_w1_parts)
};

struct EdgeBwdArgs {
  Mlp mlp;
  const int32_t* row_ptr;
  const int32_t* send;
  const int32_t* erecv;
  const int32_t* unit_r;
  const int32_t* n_units;
  const float* V;
  const float* H;
  const void* V16;
  int64_t n_owned;
  const void* Ein;      // e^k (storage type)
  const void* de_next;  // dL/de^{k+1} [E][L] in the storage type (bf16 in bf16 mode), or null (last block)
  float* dagg;          // [n_owned][L]: dL/dagg in; each receiver's sum of dz_0 out
  void* de_out;         // dL/de^k [E][L] in the storage type (may alias de_next: each row is read before it is written)
  const float* proj;    // node projections [n_local][2L] (row-split kernels), else unused
  const void* hid_in;   // streaming and row-split kernels: the forward's first-Linear ReLU output [E][L] (then layer 1 is not
                        // recomputed and hid[0] is not written), or null
  int64_t r_lo, r_hi;   // receiver range of this launch (a multiple of the planning chunk apart)
  int64_t e_base;       // first edge of the range: delta / hid rows are stored from it
  void* delta[3];
  void* hid[2];
  float* vpart;
  int nvec;
  float eps;
};

struct InGradArgs {
  Lin w1;               // first Linear of the edge MLP (backward packing)
  const int32_t* trow;  // transposed CSR over local senders
  const int32_t* tedge;
  const void* dz;       // dz_0 per edge, storage type [E][L]
  const float* dzr;     // per-receiver sums of dz_0 [n_owned][L]
  float* dv;            // [n_owned][L], accumulated into
  float* dh;            // [n_halo][L] or null
  float* dzs;           // per-sender sums of dz_0 [n_local][L]: written here, or read when dzs_ready
  int dzs_ready;
  int64_t n_local, n_owned;
};

struct DwArgs {
  const void* delta;  // d_kind 0: storage type [R][ldd]; 1: fp32 [R][ldd]
  int d_kind;
  int ldd;
  int O, I;
  int a_kind;         // 0 dense storage type, 1 dense fp32, 2 edge concat, 3 node concat,
                      // 4 node rows fp32 (owned rows a0, halo rows a2; row stride lda0),
                      // 5 node concat with the v part in bf16 (a3) and agg fp32 (a1)
  const void* a0;     // dense source / e^k / v
  int lda0;
  const float* a1;    // node concat: agg; edge concat: V (owned)
  const float* a2;    // edge concat: H (halo)
  const void* a3;     // edge concat, bf16 mode: bf16 copy of the node rows (owned then halo), or null
  const int32_t* send;
  const int32_t* erecv;
  int64_t n_owned;
  int L;
  int64_t R;
  int S;
  float* part;        // [S][O][I]
};

struct VecSeg {
  int vec_off;
  int64_t param_off;
  int len;
};

// ------------------------------------------------------------ launchers ---
hipError_t launch_zero(float* p, int64_t n, hipStream_t st);
hipError_t launch_halo_bf16(const float* H, int K, int64_t n_halo, int64_t n_owned, int L, void* V16,
                            int64_t v16_block_stride, hipStream_t st);
// p[i] -= lr * g[i] (fused multiply-add), i < n.
hipError_t launch_sgd(float* p, const float* g, int64_t n, float lr, hipStream_t st);
// nf[i][col0 + j] += out[i][j], i < n, j < d (row strides fin and d).
hipError_t launch_rollout(const float* out, int64_t n, int d, float* nf, int fin, int col0, hipStream_t st);
// Normalize: work holds norm_work_doubles(cols) doubles; cols <= NT (the
// C ABI allows at most MGN_NORM_MAX_COLS).
int norm_work_doubles(int cols);
hipError_t launch_norm_accumulate(const float* x, int64_t rows, int cols, double* stats, double* work,
                                  hipStream_t st);
hipError_t launch_norm_apply(const float* x, int64_t rows, int cols, const double* stats, double eps, float* out,
                             hipStream_t st);
// Halo exchange between partitions on one device: dst[dst_rows[i]] = (or +=,
// add != 0) src[src_rows[i]], rows of L floats (L a multiple of 4, 16-byte
// aligned rows); pairs with out-of-range indices are skipped.
hipError_t launch_rows_copy(const float* src, int64_t n_src, const int32_t* src_rows, const int32_t* dst_rows,
                            int64_t n, int L, float* dst, int64_t n_dst, int add, hipStream_t st);
hipError_t launch_pack(int prec, const float* W, int out, int in, int bwd, uint4* dst, int nkg, hipStream_t st);
hipError_t launch_erecv(const int32_t* row_ptr, int64_t n_owned, int32_t* erecv, hipStream_t st);
hipError_t launch_plan(const int32_t* row_ptr, int64_t n_owned, int te_target, int r_max, int32_t* chunk_cnt,
                       int32_t* unit_r, int32_t* n_units, hipStream_t st);
int64_t plan_max_units(int64_t n_owned, int64_t n_edges, int te_target, int r_max);
int64_t plan_chunks(int64_t n_owned);
// Receivers per planning chunk: work units never cross a multiple of it.
int plan_chunk_receivers();

// T-form row kernels (bf16, depth 2, l 64 / 128; not the decoder).  The node
// half's T-form backward needs the forward's first-Linear ReLU output
// (RowsFwdArgs::hid_out -> RowsBwdArgs::hid_in); without it the older
// row-split kernel recomputes it.
bool rows_rt(int prec, int L, int D, int kind);
// bf16, l = 256 node half and edge encoder: the streamed-weight row kernels
// (the node half's backward starts from the forward's first-Linear ReLU
// output, RowsBwdArgs::hid_in).
bool rows_rw(int prec, int L, int D, int kind);
// Whether the node half's forward keeps its first-Linear ReLU output for the
// backward (T-form or streamed-weight row kernels).
bool rows_keep_h1(int prec, int L, int D);
hipError_t launch_rows_fwd(int prec, int L, int D, int kind, const RowsFwdArgs& a, hipStream_t st);
hipError_t launch_edge_fwd(int prec, int L, int D, const EdgeFwdArgs& a, int grid, hipStream_t st);
hipError_t launch_rows_bwd(int prec, int L, int D, int kind, const RowsBwdArgs& a, int grid, hipStream_t st);
// Workgroups (= vector-partial slots) launch_rows_bwd uses when asked for `grid`.
int rows_bwd_grid(int prec, int L, int D, int kind, int grid);
// Number of per-wave partials (RowsBwdArgs::w1_part) with which the backward
// of `kind` forms its first Linear's weight gradient itself, or 0 if it
// stores delta[0] for a separate weight-gradient GEMM instead.
int rows_rt_w1_parts(int prec, int L, int D, int kind, int fin);
hipError_t launch_edge_bwd(int prec, int L, int D, const EdgeBwdArgs& a, int grid, hipStream_t st);
// Workgroups (= vector-partial slots) the edge backward uses when asked for `grid`.
int edge_bwd_grid(int prec, int L, int D, int grid);
// Whether the edge kernels take the row-split form (it needs the node
// projections of launch_node_proj for each block).
bool edge_rs(int prec, int L, int D);
hipError_t launch_node_proj(int L, const void* v16, int64_t n_local, const Lin& w1, float* proj, hipStream_t st);
// bf16, l = 256: the edge forward and backward in row-split form with the
// weights streamed through LDS (the forward, and a backward that recomputes
// h_1, need the node projections of launch_node_proj for the block).
bool edge_rsb(int prec, int L, int D);
hipError_t launch_input_grad(int prec, int L, const InGradArgs& a, hipStream_t st);
// Per-sender sums of dz_0 over the edges [e_lo, e_hi) (dz rows stored from e_lo),
// assigned (first) or added into dzs.
hipError_t launch_sender_sums(int prec, int L, const int32_t* trow, const int32_t* tedge, const void* dz, int64_t e_lo,
                              int64_t e_hi, int64_t n_local, float* dzs, int first, const int32_t* range,
                              hipStream_t st);
// range[0 .. 1] = min and max sender id of the edges [e_lo, e_hi) (empty: INT32_MAX, -1)
hipError_t launch_sender_range(const int32_t* send, int64_t e_lo, int64_t e_hi, int32_t* range, hipStream_t st);
// Register-resident weight gradient for bf16 layers with 128 inputs and 128
// outputs over many rows (dw_stream_ok); part needs dw_stream_parts() * 16384
// floats; writes (or adds to) dst[o * ldw + i].
int dw_stream_parts();
bool dw_stream_ok(int prec, const DwArgs& a);
hipError_t launch_dw_stream(const DwArgs& a, float* dst, int ldw, int accumulate, hipStream_t st);
// The same for bf16 layers with 256 inputs and 256 outputs in one launch (each
// operand row read once; same partial buffer).
bool dw_stream_quad_ok(int prec, const DwArgs& a);
hipError_t launch_dw_stream_quad(const DwArgs& a, float* dst, int ldw, int accumulate, hipStream_t st);
// The same for fp32 layers with 128 inputs and 128 outputs (dw_stream_f32_ok):
// wave partials in plain [o][i] order, then the fixed-order split reduction.
bool dw_stream_f32_ok(int prec, const DwArgs& a);
hipError_t launch_dw_stream_f32(const DwArgs& a, float* dst, int ldw, int accumulate, hipStream_t st);
hipError_t launch_dw(int prec, const DwArgs& a, hipStream_t st);
hipError_t launch_dw_reduce(const float* part, int S, int O, int I, float* dst, int ldw, int accumulate,
                            hipStream_t st);
hipError_t launch_vec_reduce(const float* vpart, int nwg, int nvec, const VecSeg* segs, int nseg, float* dparams,
                             int accumulate, hipStream_t st);
// Masked MSE and its gradient; the mean is over global_rows rows when > 0,
// else over this call's masked rows.
hipError_t launch_mse(const float* out, const float* target, const uint8_t* mask, int64_t n, int d,
                      int64_t global_rows, float* loss, float* d_out, hipStream_t st);

// tile sizes the host needs to know (rows per edge sub-tile, per prec/L/D)
int edge_tile_rows(int prec, int L, int D);
int dw_splits(int64_t R, int O, int I);

}  // namespace mgn

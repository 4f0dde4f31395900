// libmgn C ABI (include/mgn.h): model state, parameter layout and packing,
// argument / state checks, workspace plan and the launch sequence of one
// training step.  Device work is enqueued on the caller's stream; the only
// synchronising calls are the parameter copies and graph validation.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <string>
#include <vector>

#include "kernels.h"
#include "mgn_internal.h"

using namespace mgn;

namespace {

thread_local std::string g_err;  // last error of calls without a model

constexpr int BWD_GRID = 1024;   // fixed persistent grid of the backward kernels (multiple of 8)
constexpr int FWD_EDGE_GRID = 2048;

struct LinL {
  int64_t w = 0, b = 0;  // parameter offsets
  int in = 0, out = 0;
  size_t pf = 0, pb = 0;  // packed offsets (uint4 units)
  int nkgf = 0, nkgb = 0;
};

struct MlpL {
  LinL lin[3];
  int64_t gamma = -1, beta = -1;
  int depth = 0;
  int nvec = 0;  // bias + LayerNorm gradient entries: (depth-1)*l + out + (LN ? 2l : 0)
};

struct WsPlan {
  size_t erecv, chunk, unit_r, nunits, V, V16, PROJ, AGG, ES, DV[2], DAGG, DZS, DE, DEL_E[3], HID_E[2], DEL_N[3], HID_N[2],
      HID_NK, HID_E1, PART, VPART, SRANGE, total;
  int64_t max_units;
  // edge-stream checkpointing: interval s (0: every block kept), checkpoints
  bool lean = false;
  int s = 0, nck = 0;
  // forward-only plan (inference): working copies only, no backward buffers
  bool infer = false;
  // node projections kept per block (row-split kernels, every block kept)
  bool proj_all = false;
  // blocks k >= h1_first keep their first-Linear ReLU output (HID_E1 slot k - h1_first)
  int h1_first = 0;
  // receiver / edge boundaries of the backward's edge chunks
  std::vector<int64_t> cr, ce;
};

constexpr int64_t LEAN_CHUNK_EDGES = 8 << 20;  // edges per backward chunk with checkpointing

}  // namespace

struct mgn_model {
  mgn_config cfg{};
  int prec = 0, L = 0, K = 0, D = 0;
  int kg = 16;  // k-group of the precision
  std::vector<MlpL> mlp;  // enc_node, enc_edge, {edge_k, node_k}..., dec
  int64_t P = 0;
  float* params = nullptr;
  uint4* packed = nullptr;
  size_t packed_n = 0;
  bool params_set = false;
  // graph accepted by mgn_graph_validate, and a host copy of its row_ptr
  bool graph_ok = false;
  mgn_graph vg{};
  std::vector<int32_t> rp_host;
  int ckpt = 0;                 // edge-stream checkpoint interval (0: keep every block)
  int h1_stash = 0;             // row-split kernels: blocks whose first-Linear ReLU output the forward keeps
  bool infer = false;           // forward-only plan (mgn_set_inference)
  int64_t chunk_edges = 0;      // edges per backward chunk with checkpointing (0: the default)
  // what the last forward used (kept for the backward)
  bool fwd_done = false;
  // checkpointing: the forward's last block left its aggregate in its slot,
  // and no backward block has run since (the backward's last block reads it
  // instead of running that block's edge forward once more)
  bool agg_last = false;
  mgn_graph g{};
  const float *nf = nullptr, *ef = nullptr, *halo = nullptr;
  float* out = nullptr;
  char* ws = nullptr;
  WsPlan plan{};
  // staged step: the forward's next block (-1: no forward in progress); the
  // backward in progress, its next block (-1: its blocks are done), the dL/dv
  // buffer holding the gradient of the last stage's node latents, and the
  // gradient outputs of the backward_begin call
  int fwd_next = -1;
  bool bwd_active = false;
  int bwd_next = -1, bwd_a = 0;
  float* d_params = nullptr;
  float* d_halo = nullptr;
  int accumulate = 0;
  std::string err;
  // launch timing
  bool timing = false;
  std::vector<hipEvent_t> ev_pool;
  size_t ev_used = 0;
  std::vector<std::pair<int, size_t>> ev_rec;  // (timer, index of the start event)

  MlpL& enc_node() { return mlp[0]; }
  MlpL& enc_edge() { return mlp[1]; }
  MlpL& edge(int k) { return mlp[2 + 2 * k]; }
  MlpL& node(int k) { return mlp[3 + 2 * k]; }
  MlpL& dec() { return mlp.back(); }
};

namespace {

mgn_status fail(mgn_model* m, mgn_status s, const std::string& msg) {
  if (m)
    m->err = msg;
  else
    g_err = msg;
  return s;
}

mgn_status hip_fail(mgn_model* m, hipError_t e, const char* what) {
  return fail(m, MGN_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

}  // namespace

mgn_status mgn::set_error(mgn_model* m, mgn_status s, const std::string& msg) { return fail(m, s, msg); }
bool mgn::timing_enabled(const mgn_model* m) { return m && m->timing; }

namespace {

// Refreshes the packed copies of every Linear's weights from the fp32 master copy.
hipError_t repack(mgn_model* m, hipStream_t st) {
  for (const MlpL& ml : m->mlp)
    for (int j = 0; j < ml.depth; ++j) {
      const LinL& L = ml.lin[j];
      hipError_t e = launch_pack(m->prec, m->params + L.w, L.out, L.in, 0, m->packed + L.pf, L.nkgf, st);
      if (e == hipSuccess) e = launch_pack(m->prec, m->params + L.w, L.out, L.in, 1, m->packed + L.pb, L.nkgb, st);
      if (e != hipSuccess) return e;
    }
  return hipSuccess;
}

size_t tsize(const mgn_model* m) { return m->prec == BF16 ? 2 : 4; }

// Records a pair of events around the launches in its scope when timing is on.
struct Timed {
  mgn_model* m;
  hipStream_t st;
  size_t i0 = 0;
  bool on;
  hipEvent_t next() {
    if (m->ev_used == m->ev_pool.size()) {
      hipEvent_t e;
      if (hipEventCreate(&e) != hipSuccess) return nullptr;
      m->ev_pool.push_back(e);
    }
    return m->ev_pool[m->ev_used++];
  }
  Timed(mgn_model* m_, int timer, hipStream_t s) : m(m_), st(s), on(m_->timing) {
    if (!on) return;
    i0 = m->ev_used;
    hipEvent_t a = next(), b = next();
    if (!a || !b) {
      on = false;
      return;
    }
    (void)hipEventRecord(a, st);
    m->ev_rec.push_back({timer, i0});
  }
  ~Timed() {
    if (on) (void)hipEventRecord(m->ev_pool[i0 + 1], st);
  }
};

MlpL make_mlp(mgn_model* m, int fin, int fout, bool ln, int64_t& off, size_t& poff) {
  MlpL r;
  r.depth = m->D;
  int prev = fin;
  for (int j = 0; j < m->D; ++j) {
    LinL& L = r.lin[j];
    L.in = prev;
    L.out = (j == m->D - 1) ? fout : m->L;
    L.w = off;
    L.b = off + (int64_t)L.out * L.in;
    off += (int64_t)L.out * L.in + L.out;
    L.nkgf = (L.in + m->kg - 1) / m->kg;
    L.nkgb = (L.out + m->kg - 1) / m->kg;
    L.pf = poff;
    poff += (size_t)((L.out + 15) / 16) * L.nkgf * 64;
    L.pb = poff;
    poff += (size_t)((L.in + 15) / 16) * L.nkgb * 64;
    prev = L.out;
  }
  if (ln) {
    r.gamma = off;
    r.beta = off + fout;
    off += 2 * (int64_t)fout;
  }
  r.nvec = (m->D - 1) * m->L + fout + (ln ? 2 * fout : 0);
  return r;
}

Mlp dev_mlp(const mgn_model* m, const MlpL& l) {
  Mlp d{};
  d.depth = l.depth;
  for (int j = 0; j < l.depth; ++j) {
    const LinL& L = l.lin[j];
    d.lin[j] = Lin{m->packed + L.pf, m->packed + L.pb, m->params + L.b, L.in, L.out, L.nkgf, L.nkgb};
  }
  d.gamma = l.gamma >= 0 ? m->params + l.gamma : nullptr;
  d.beta = l.beta >= 0 ? m->params + l.beta : nullptr;
  return d;
}

size_t al(size_t x) { return (x + 255) & ~(size_t)255; }

bool same_graph(const mgn_graph& a, const mgn_graph& b) {
  return a.n_owned == b.n_owned && a.n_halo == b.n_halo && a.n_edges == b.n_edges && a.row_ptr == b.row_ptr &&
         a.send == b.send && a.trow_ptr == b.trow_ptr && a.tedge == b.tedge;
}

WsPlan make_plan(const mgn_model* m, const mgn_graph* g) {
  WsPlan p{};
  const int64_t no = g->n_owned, ne = g->n_edges, nl = no + g->n_halo, L = m->L, K = m->K;
  const size_t ts = tsize(m);
  const int te = edge_tile_rows(m->prec, m->L, m->D);
  p.max_units = plan_max_units(no, ne, 4 * te, 4 * te);
  p.infer = m->infer;
  p.lean = m->ckpt > 0 && K > 0 && !p.infer;
  p.s = m->ckpt;
  p.nck = p.lean ? (int)((K + p.s - 1) / p.s) : 0;
  // backward edge chunks: one, or ~LEAN_CHUNK_EDGES edges each on planning-chunk receiver boundaries
  p.cr = {0};
  const int64_t che = m->chunk_edges > 0 ? m->chunk_edges : LEAN_CHUNK_EDGES;
  const bool host_rp = (int64_t)m->rp_host.size() == no + 1 && same_graph(*g, m->vg);
  if (p.lean && ne > che && host_rp) {
    const int64_t nc = (ne + che - 1) / che, q = plan_chunk_receivers();
    for (int64_t c = 1; c < nc; ++c) {
      const int64_t target = ne * c / nc;
      int64_t r = std::lower_bound(m->rp_host.begin(), m->rp_host.end(), (int32_t)target) - m->rp_host.begin();
      r = r / q * q;
      if (r > p.cr.back() && r < no) p.cr.push_back(r);
    }
  }
  p.cr.push_back(no);
  int64_t emax = 0;
  for (int64_t r : p.cr) p.ce.push_back(r == no ? ne : (host_rp ? m->rp_host[r] : 0));
  for (size_t c = 0; c + 1 < p.ce.size(); ++c) emax = std::max(emax, p.ce[c + 1] - p.ce[c]);
  size_t o = 0;
  auto take = [&](size_t bytes) {
    size_t r = o;
    o += al(bytes);
    return r;
  };
  p.erecv = take(4 * (size_t)ne);
  p.chunk = take(4 * (size_t)plan_chunks(no));
  p.unit_r = take(4 * (size_t)(p.max_units + 1));
  p.nunits = take(4);
  const bool one = p.lean || p.infer;  // one working slot per block-level buffer
  // fp32 node stream: every block's input, or (checkpointing, inference) two working rows
  p.V = take(4 * (size_t)(one ? 2 : K + 1) * no * L);
  // bf16 mode: bf16 copy of every block's node input (inference: two), owned then halo rows
  p.V16 = m->prec == BF16 ? take(2 * (size_t)(p.infer ? 2 : K + 1) * nl * L) : 0;
  // row-split edge kernels: blocks whose first-Linear ReLU output the forward
  // keeps (the last h1_stash of them, as memory allows) and whose backward
  // therefore reads neither e^k's first-layer recompute nor the projections
  int64_t nh1 = 0;
  if (!p.infer && !p.lean && K > 0) nh1 = edge_rs(m->prec, m->L, m->D) ? std::min<int64_t>(m->h1_stash, K) : K;
  p.h1_first = (int)(K - nh1);
  // row-split edge kernels: node projections of every block's input that the
  // backward recomputes from (blocks before h1_first) plus one slot shared by
  // the stashed blocks' forwards, or of the current block only
  // (checkpointing, inference)
  p.proj_all = edge_rs(m->prec, m->L, m->D) && !one;
  p.PROJ = edge_rs(m->prec, m->L, m->D) ? take(4 * (size_t)(one ? 1 : p.h1_first + (nh1 > 0)) * nl * 2 * L)
           : edge_rsb(m->prec, m->L, m->D) ? take(4 * (size_t)nl * 2 * L)  // l = 256 forward: the current block's
           : 0;
  // aggregated messages: every block's; (checkpointing) two slots, block k's
  // in slot k % 2, so that the backward's recompute of e^k leaves agg^{k-1}
  // in place for the next block; (inference) one
  p.AGG = take(4 * (size_t)(p.infer ? 1 : p.lean ? 2 : K) * no * L);
  // edge stream: every block's input, the checkpoints plus one working copy,
  // or (inference) one copy updated in place
  p.ES = take(ts * (size_t)(p.infer ? 1 : p.lean ? p.nck + 1 : std::max<int64_t>(K, 1)) * ne * L);
  // streaming edge kernels, every block kept: each block's first-Linear ReLU
  // output, written by the forward, so the backward skips recomputing the
  // first Linear (half its products) and the row gather
  // (row-split kernels: for the last h1_stash blocks only, as memory allows;
  // the others recompute it from e and the kept projections)
  p.HID_E1 = nh1 > 0 ? take(ts * (size_t)nh1 * ne * L) : 0;
  if (p.infer) {
    p.total = o;
    return p;
  }
  p.DV[0] = take(4 * (size_t)no * L);
  p.DV[1] = take(4 * (size_t)no * L);
  p.DAGG = take(4 * (size_t)no * L);
  p.DZS = take(4 * (size_t)nl * L);
  p.DE = take(ts * (size_t)ne * L);  // dL/de in the storage type, updated in place block by block
  for (int j = 0; j < 3; ++j) p.DEL_E[j] = j < m->D ? take(ts * (size_t)emax * L) : 0;
  for (int j = 0; j < 2; ++j) p.HID_E[j] = j < m->D - 1 ? take(ts * (size_t)emax * L) : 0;
  for (int j = 0; j < 3; ++j) p.DEL_N[j] = j < m->D ? take(ts * (size_t)no * std::max<int64_t>(L, 16)) : 0;
  for (int j = 0; j < 2; ++j) p.HID_N[j] = j < m->D - 1 ? take(ts * (size_t)no * L) : 0;
  // T-form node kernels: every block's first-Linear ReLU output, written by
  // the forward for the backward; checkpointing: one block's, recomputed
  p.HID_NK = rows_keep_h1(m->prec, L, m->D) ? take(2 * (size_t)(p.lean ? 1 : K) * no * L) : 0;
  // split-K partials: the largest S*O*I over all weight matrices
  size_t part = 0;
  const size_t nm = m->mlp.size();
  for (size_t i = 0; i < nm; ++i) {
    const MlpL& ml = m->mlp[i];
    // EncEdge (index 1) and the edge MLPs (even indices 2 .. nm-2) run over edges
    const bool edge_rows = i == 1 || (i >= 2 && i + 1 < nm && i % 2 == 0);
    const int64_t R = edge_rows ? ne : nl;
    for (int j = 0; j < ml.depth; ++j) {
      const LinL& Ln = ml.lin[j];
      part = std::max(part, (size_t)dw_splits(R, Ln.out, Ln.in) * Ln.out * Ln.in);
    }
  }
  part = std::max(part, (size_t)dw_stream_parts() * 16384);
  p.PART = take(4 * part);
  int nvec = 0;
  for (const MlpL& ml : m->mlp) nvec = std::max(nvec, ml.nvec);
  p.VPART = take(4 * (size_t)BWD_GRID * nvec);
  p.SRANGE = take(8);  // sender-id range of a backward edge chunk
  p.total = o;
  return p;
}


bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

mgn_status check_graph_args(mgn_model* m, const mgn_graph* g) {
  if (!g) return fail(m, MGN_E_ARG, "graph is NULL");
  if (g->n_owned < 0 || g->n_halo < 0 || g->n_edges < 0)
    return fail(m, MGN_E_ARG, "graph sizes must be non-negative");
  if (g->n_owned + g->n_halo > INT32_MAX || g->n_edges > INT32_MAX)
    return fail(m, MGN_E_UNSUPPORTED, "graph larger than int32 indexing");
  if (!g->row_ptr || !g->trow_ptr || (g->n_edges > 0 && (!g->send || !g->tedge)))
    return fail(m, MGN_E_ARG, "graph array is NULL");
  if (!aligned(g->row_ptr, 4) || !aligned(g->send, 4) || !aligned(g->trow_ptr, 4) || !aligned(g->tedge, 4))
    return fail(m, MGN_E_ARG, "graph arrays must be 4-byte aligned");
  return MGN_OK;
}

}  // namespace

// ================================================================== ABI ===
extern "C" {

const char* mgn_last_error(const mgn_model* m) { return m ? m->err.c_str() : g_err.c_str(); }

mgn_status mgn_create(const mgn_config* cfg, mgn_model** out) {
  if (!cfg || !out) return fail(nullptr, MGN_E_ARG, "mgn_create: NULL argument");
  *out = nullptr;
  const mgn_config& c = *cfg;
  if (c.latent != 64 && c.latent != 128 && c.latent != 256)
    return fail(nullptr, MGN_E_UNSUPPORTED, "latent must be 64, 128 or 256");
  if (c.depth != 2 && c.depth != 3) return fail(nullptr, MGN_E_UNSUPPORTED, "depth must be 2 or 3");
  if (c.n_blocks < 0 || c.n_blocks > 1024) return fail(nullptr, MGN_E_UNSUPPORTED, "n_blocks must be 0..1024");
  if (c.node_in < 1 || c.node_in > 32 || c.edge_in < 1 || c.edge_in > 32)
    return fail(nullptr, MGN_E_UNSUPPORTED, "node_in and edge_in must be 1..32");
  if (c.node_out < 1 || c.node_out > 16) return fail(nullptr, MGN_E_UNSUPPORTED, "node_out must be 1..16");
  if (c.precision != MGN_FP32 && c.precision != MGN_BF16)
    return fail(nullptr, MGN_E_UNSUPPORTED, "precision must be MGN_FP32 or MGN_BF16");
  if (!(c.ln_eps > 0.f)) return fail(nullptr, MGN_E_ARG, "ln_eps must be positive");
  mgn_model* m = new mgn_model();
  m->cfg = c;
  m->prec = c.precision == MGN_BF16 ? BF16 : F32;
  m->L = c.latent;
  m->K = c.n_blocks;
  m->D = c.depth;
  m->kg = m->prec == BF16 ? PBF16::KG : PF32::KG;
  int64_t off = 0;
  size_t poff = 0;
  m->mlp.push_back(make_mlp(m, c.node_in, m->L, true, off, poff));
  m->mlp.push_back(make_mlp(m, c.edge_in, m->L, true, off, poff));
  for (int k = 0; k < m->K; ++k) {
    m->mlp.push_back(make_mlp(m, 3 * m->L, m->L, true, off, poff));
    m->mlp.push_back(make_mlp(m, 2 * m->L, m->L, true, off, poff));
  }
  m->mlp.push_back(make_mlp(m, m->L, c.node_out, false, off, poff));
  m->P = off;
  m->packed_n = poff;
  *out = m;  // device memory is allocated by the first mgn_set_params
  return MGN_OK;
}

void mgn_destroy(mgn_model* m) {
  if (!m) return;
  for (hipEvent_t e : m->ev_pool) (void)hipEventDestroy(e);
  if (m->params) (void)hipFree(m->params);
  if (m->packed) (void)hipFree(m->packed);
  delete m;
}

int64_t mgn_param_count(const mgn_model* m) { return m ? m->P : -1; }

mgn_status mgn_set_params(mgn_model* m, const float* src, int src_on_device, mgn_stream stream) {
  if (!m) return fail(nullptr, MGN_E_ARG, "mgn_set_params: model is NULL");
  if (!src) return fail(m, MGN_E_ARG, "mgn_set_params: src is NULL");
  hipStream_t st = (hipStream_t)stream;
  if (!m->params) {
    hipError_t a = hipMalloc(&m->params, sizeof(float) * m->P);
    if (a == hipSuccess) a = hipMalloc(&m->packed, sizeof(uint4) * m->packed_n);
    if (a != hipSuccess) {
      if (m->params) (void)hipFree(m->params);
      m->params = nullptr;
      m->packed = nullptr;
      return fail(m, MGN_E_NOMEM, std::string("mgn_set_params: ") + hipGetErrorString(a));
    }
  }
  hipError_t e = hipMemcpyAsync(m->params, src, sizeof(float) * m->P,
                                src_on_device ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice, st);
  if (e != hipSuccess) return hip_fail(m, e, "mgn_set_params copy");
  e = repack(m, st);
  if (e != hipSuccess) return hip_fail(m, e, "mgn_set_params pack");
  e = hipStreamSynchronize(st);
  if (e != hipSuccess) return hip_fail(m, e, "mgn_set_params sync");
  m->params_set = true;
  m->fwd_done = false;  // a step in progress is dropped
  m->fwd_next = -1;
  m->bwd_active = false;
  return MGN_OK;
}

mgn_status mgn_sgd_step(mgn_model* m, const float* grad, float lr, mgn_stream stream) {
  if (!m) return fail(nullptr, MGN_E_ARG, "mgn_sgd_step: model is NULL");
  if (!grad || !aligned(grad, 4)) return fail(m, MGN_E_ARG, "mgn_sgd_step: grad NULL or misaligned");
  if (!std::isfinite(lr)) return fail(m, MGN_E_ARG, "mgn_sgd_step: learning rate is not finite");
  if (!m->params_set) return fail(m, MGN_E_STATE, "mgn_sgd_step: parameters were never set");
  hipStream_t st = (hipStream_t)stream;
  m->fwd_done = false;  // the parameters change: a step in progress is dropped
  m->fwd_next = -1;
  m->bwd_active = false;
  hipError_t e = launch_sgd(m->params, grad, m->P, lr, st);
  if (e == hipSuccess) e = repack(m, st);
  if (e != hipSuccess) return hip_fail(m, e, "mgn_sgd_step");
  return MGN_OK;
}

mgn_status mgn_get_params(const mgn_model* cm, float* dst, int dst_on_device, mgn_stream stream) {
  mgn_model* m = const_cast<mgn_model*>(cm);
  if (!m) return fail(nullptr, MGN_E_ARG, "mgn_get_params: model is NULL");
  if (!dst) return fail(m, MGN_E_ARG, "mgn_get_params: dst is NULL");
  if (!m->params_set) return fail(m, MGN_E_STATE, "mgn_get_params: parameters were never set");
  hipStream_t st = (hipStream_t)stream;
  hipError_t e = hipMemcpyAsync(dst, m->params, sizeof(float) * m->P,
                                dst_on_device ? hipMemcpyDeviceToDevice : hipMemcpyDeviceToHost, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e != hipSuccess) return hip_fail(m, e, "mgn_get_params");
  return MGN_OK;
}

mgn_status mgn_partition_slabs(const int32_t* key, int64_t n, int32_t nparts, int32_t* part) {
  return partition_slabs(key, n, nparts, part, g_err);
}

mgn_status mgn_graph_sizes(const int32_t* send, const int32_t* recv, int64_t n_edges, const int32_t* part,
                           int64_t n_nodes, int32_t p, int64_t* sizes) {
  return graph_sizes(send, recv, n_edges, part, n_nodes, p, sizes, g_err);
}

mgn_status mgn_graph_build(const int32_t* send, const int32_t* recv, int64_t n_edges, const int32_t* part,
                           int64_t n_nodes, int32_t p, int32_t* row_ptr, int32_t* send_local, int32_t* eperm,
                           int32_t* trow_ptr, int32_t* tedge, int32_t* l2g) {
  return graph_build(send, recv, n_edges, part, n_nodes, p, row_ptr, send_local, eperm, trow_ptr, tedge, l2g, g_err);
}

mgn_status mgn_graph_validate(mgn_model* m, const mgn_graph* g, mgn_stream stream) {
  if (!m) return fail(nullptr, MGN_E_ARG, "mgn_graph_validate: model is NULL");
  mgn_status s = check_graph_args(m, g);
  if (s) return s;
  const int64_t no = g->n_owned, nh = g->n_halo, ne = g->n_edges, nl = no + nh;
  std::vector<int32_t> rp(no + 1), snd(ne), tr(nl + 1), te(ne);
  hipStream_t st = (hipStream_t)stream;
  hipError_t e = hipStreamSynchronize(st);
  if (e == hipSuccess) e = hipMemcpy(rp.data(), g->row_ptr, 4 * (no + 1), hipMemcpyDeviceToHost);
  if (e == hipSuccess && ne) e = hipMemcpy(snd.data(), g->send, 4 * ne, hipMemcpyDeviceToHost);
  if (e == hipSuccess) e = hipMemcpy(tr.data(), g->trow_ptr, 4 * (nl + 1), hipMemcpyDeviceToHost);
  if (e == hipSuccess && ne) e = hipMemcpy(te.data(), g->tedge, 4 * ne, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(m, e, "mgn_graph_validate copy");
  std::string err;
  s = graph_check(no, nh, ne, rp.data(), snd.data(), tr.data(), te.data(), err);
  if (s) return fail(m, s, err);
  m->vg = *g;
  m->graph_ok = true;
  m->rp_host = std::move(rp);
  return MGN_OK;
}

mgn_status mgn_set_recompute(mgn_model* m, int32_t interval, int64_t chunk_edges) {
  if (!m) return fail(nullptr, MGN_E_ARG, "mgn_set_recompute: model is NULL");
  if (interval < 0 || chunk_edges < 0) return fail(m, MGN_E_ARG, "mgn_set_recompute: negative argument");
  if (interval > 0 && m->prec != BF16)
    return fail(m, MGN_E_UNSUPPORTED, "mgn_set_recompute: edge-stream checkpointing needs the bf16 precision");
  m->ckpt = interval;
  m->chunk_edges = chunk_edges;
  m->fwd_done = false;  // the workspace plan changes: a step in progress is dropped
  m->fwd_next = -1;
  m->bwd_active = false;
  return MGN_OK;
}

mgn_status mgn_set_h1_stash(mgn_model* m, int32_t n_blocks) {
  if (!m) return fail(nullptr, MGN_E_ARG, "mgn_set_h1_stash: model is NULL");
  if (n_blocks < 0) return fail(m, MGN_E_ARG, "mgn_set_h1_stash: negative block count");
  m->h1_stash = n_blocks;
  m->fwd_done = false;  // the workspace plan changes: a step in progress is dropped
  m->fwd_next = -1;
  m->bwd_active = false;
  return MGN_OK;
}

mgn_status mgn_set_inference(mgn_model* m, int32_t on) {
  if (!m) return fail(nullptr, MGN_E_ARG, "mgn_set_inference: model is NULL");
  m->infer = on != 0;
  m->fwd_done = false;  // the workspace plan changes: a step in progress is dropped
  m->fwd_next = -1;
  m->bwd_active = false;
  return MGN_OK;
}

mgn_status mgn_rollout_update(const float* out, int64_t n, int32_t node_out, float* node_feat, int32_t node_in,
                              int32_t col0, mgn_stream stream) {
  if (n < 0 || node_out < 1 || node_in < 1 || col0 < 0 || col0 + node_out > node_in)
    return fail(nullptr, MGN_E_ARG, "mgn_rollout_update: bad sizes (need col0 + node_out <= node_in)");
  if (n == 0) return MGN_OK;
  if (!out || !node_feat || !aligned(out, 4) || !aligned(node_feat, 4))
    return fail(nullptr, MGN_E_ARG, "mgn_rollout_update: NULL or misaligned pointer");
  hipError_t e = launch_rollout(out, n, node_out, node_feat, node_in, col0, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(nullptr, e, "mgn_rollout_update");
  return MGN_OK;
}

mgn_status mgn_norm_accumulate(const float* x, int64_t rows, int32_t cols, double* stats, double* work,
                               mgn_stream stream) {
  if (rows < 0 || cols < 1 || cols > MGN_NORM_MAX_COLS)
    return fail(nullptr, MGN_E_ARG, "mgn_norm_accumulate: bad sizes (rows >= 0, 1 <= cols <= MGN_NORM_MAX_COLS)");
  if (!stats || !work || !aligned(stats, 8) || !aligned(work, 8) || (rows > 0 && (!x || !aligned(x, 4))))
    return fail(nullptr, MGN_E_ARG, "mgn_norm_accumulate: NULL or misaligned pointer");
  if (rows == 0) return MGN_OK;
  hipError_t e = launch_norm_accumulate(x, rows, cols, stats, work, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(nullptr, e, "mgn_norm_accumulate");
  return MGN_OK;
}

mgn_status mgn_norm_apply(const float* x, int64_t rows, int32_t cols, const double* stats, double eps, float* out,
                          mgn_stream stream) {
  if (rows < 0 || cols < 1 || cols > MGN_NORM_MAX_COLS || !(eps > 0))
    return fail(nullptr, MGN_E_ARG, "mgn_norm_apply: bad sizes or eps (rows >= 0, 1 <= cols <= MGN_NORM_MAX_COLS, eps > 0)");
  if (!stats || !aligned(stats, 8) || (rows > 0 && (!x || !out || !aligned(x, 4) || !aligned(out, 4))))
    return fail(nullptr, MGN_E_ARG, "mgn_norm_apply: NULL or misaligned pointer");
  if (rows == 0) return MGN_OK;
  hipError_t e = launch_norm_apply(x, rows, cols, stats, eps, out, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(nullptr, e, "mgn_norm_apply");
  return MGN_OK;
}

mgn_status mgn_workspace_size(const mgn_model* cm, const mgn_graph* g, size_t* bytes) {
  mgn_model* m = const_cast<mgn_model*>(cm);
  if (!m) return fail(nullptr, MGN_E_ARG, "mgn_workspace_size: model is NULL");
  if (!bytes) return fail(m, MGN_E_ARG, "mgn_workspace_size: bytes is NULL");
  mgn_status s = check_graph_args(m, g);
  if (s) return s;
  *bytes = make_plan(m, g).total;
  return MGN_OK;
}

}  // extern "C"

namespace {

// Block k's first-Linear ReLU output slot (`bytes` per block), or null when
// the plan keeps none for it.
void* h1_slot(const WsPlan& p, char* ws, int k, size_t bytes) {
  return p.HID_E1 && k >= p.h1_first ? (void*)(ws + p.HID_E1 + bytes * (size_t)(k - p.h1_first)) : nullptr;
}

// Node projections of block k (one shared slot when checkpointing, and one
// shared by the blocks k >= h1_first, whose backward does not read them).
float* proj_block(const WsPlan& p, char* ws, int k, int64_t nl, int L) {
  return (float*)(ws + p.PROJ) + (p.proj_all ? (size_t)std::min(k, p.h1_first) * nl * 2 * L : 0);
}

// The edge half of block k forward: node projections (row-split path), then
// the fused edge kernel: e^{k+1} = e^k + m into eout (may equal ein, or be
// null), ordered receiver sums into agg.
hipError_t edge_forward_block(mgn_model* m, const mgn_graph& g, const WsPlan& p, char* ws, const float* halo, int k,
                              float* v, void* v16, const void* ein, void* eout, float* agg, hipStream_t st) {
  const int64_t no = g.n_owned, nh = g.n_halo;
  const int L = m->L, D = m->D;
  if (no == 0) return hipSuccess;
  EdgeFwdArgs ea{};
  ea.mlp = dev_mlp(m, m->edge(k));
  ea.row_ptr = g.row_ptr;
  ea.send = g.send;
  ea.erecv = (int32_t*)(ws + p.erecv);
  ea.unit_r = (int32_t*)(ws + p.unit_r);
  ea.n_units = (int32_t*)(ws + p.nunits);
  ea.V = v;
  ea.H = nh > 0 ? halo + (size_t)k * nh * L : nullptr;
  ea.V16 = v16;
  ea.n_owned = no;
  ea.Ein = ein;
  ea.Eout = eout;
  ea.agg = agg;
  ea.eps = m->cfg.ln_eps;
  ea.hid_out = h1_slot(p, ws, k, tsize(m) * (size_t)g.n_edges * L);
  const bool rs = edge_rs(m->prec, L, D) || edge_rsb(m->prec, L, D);
  float* proj = rs ? proj_block(p, ws, k, no + nh, L) : nullptr;
  ea.proj = proj;
  hipError_t e = hipSuccess;
  if (rs) {
    Timed t_(m, MGN_T_NODE_PROJ, st);
    e = launch_node_proj(L, v16, no + nh, ea.mlp.lin[0], proj, st);
    if (e != hipSuccess) return e;
  }
  Timed t_(m, MGN_T_EDGE_FWD, st);
  return launch_edge_fwd(m->prec, L, D, ea, FWD_EDGE_GRID, st);
}

}  // namespace

namespace {

// Weight gradient of Linear j of an MLP: split-K GEMM into the partial
// buffer, then the fixed-order reduction into d_params.
// Gradient of Linear L's weight, or of its input columns [col0, col0 + ncols)
// when ncols >= 0 (the operand a then covers just those columns).
hipError_t run_dw(mgn_model* m, const LinL& L, DwArgs a, float* d_params, int accumulate, hipStream_t st,
                  int col0 = 0, int ncols = -1) {
  a.O = L.out;
  a.I = ncols < 0 ? L.in : ncols;
  a.S = dw_splits(a.R, a.O, a.I);
  a.part = (float*)(m->ws + m->plan.PART);
  a.L = m->L;
  float* dst = d_params + L.w + col0;
  if (a.R == 0) {
    // no rows: the gradient is zero
    if (accumulate) return hipSuccess;
    if (ncols < 0) return launch_zero(dst, (int64_t)L.out * L.in, st);
    for (int o = 0; o < L.out; ++o) {
      hipError_t e = launch_zero(dst + (size_t)o * L.in, a.I, st);
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  }
  Timed t_(m, MGN_T_WEIGHT_GRAD, st);
  if (dw_stream_ok(m->prec, a)) return launch_dw_stream(a, dst, L.in, accumulate, st);
  if (dw_stream_quad_ok(m->prec, a)) return launch_dw_stream_quad(a, dst, L.in, accumulate, st);
  if (dw_stream_f32_ok(m->prec, a)) return launch_dw_stream_f32(a, dst, L.in, accumulate, st);
  if ((a.O > 128 || a.I > 128) && a.O % 128 == 0 && a.I % 128 == 0) {
    // wider layers (l = 256) as 128 x 128 blocks on the register-resident
    // kernels: each block re-reads its column ranges of both operands
    DwArgs q = a;
    q.O = 128;
    q.I = 128;
    const bool bf = dw_stream_ok(m->prec, q), f32 = dw_stream_f32_ok(m->prec, q);
    if (bf || f32) {
      const size_t st_sz = tsize(m);
      const size_t ds = a.d_kind == 1 ? 4 : st_sz, as = a.a_kind == 1 ? 4 : st_sz;
      for (int o0 = 0; o0 < a.O; o0 += 128)
        for (int i0 = 0; i0 < a.I; i0 += 128) {
          q.delta = (const char*)a.delta + ds * o0;
          q.a0 = (const char*)a.a0 + as * i0;
          float* qd = dst + (size_t)o0 * L.in + i0;
          hipError_t e = bf ? launch_dw_stream(q, qd, L.in, accumulate, st)
                            : launch_dw_stream_f32(q, qd, L.in, accumulate, st);
          if (e != hipSuccess) return e;
        }
      return hipSuccess;
    }
  }
  hipError_t e = launch_dw(m->prec, a, st);
  if (e == hipSuccess) e = launch_dw_reduce(a.part, a.S, a.O, a.I, dst, L.in, accumulate, st);
  return e;
}

hipError_t run_vec(mgn_model* m, const MlpL& ml, float* d_params, int accumulate, hipStream_t st,
                   int slots = BWD_GRID) {
  VecSeg segs[4];
  int n = 0, off = 0;
  for (int j = 0; j < ml.depth; ++j) {
    segs[n++] = VecSeg{off, ml.lin[j].b, ml.lin[j].out};
    off += (j + 1 < ml.depth) ? m->L : ml.lin[j].out;
  }
  if (ml.gamma >= 0) segs[n++] = VecSeg{off, ml.gamma, 2 * ml.lin[ml.depth - 1].out};
  Timed t_(m, MGN_T_WEIGHT_GRAD, st);
  return launch_vec_reduce((float*)(m->ws + m->plan.VPART), slots, ml.nvec, segs, n, d_params, accumulate, st);
}

}  // namespace

namespace {

// Views of the buffers of the model's current step (the plan, workspace and
// graph recorded by the forward's first stage).
struct Views {
  const WsPlan& p;
  char* ws;
  int64_t no, nh, ne;
  int L;
  size_t ts;
  bool bf16;
  explicit Views(const mgn_model* m)
      : p(m->plan), ws(m->ws), no(m->g.n_owned), nh(m->g.n_halo), ne(m->g.n_edges), L(m->L), ts(tsize(m)),
        bf16(m->prec == BF16) {}
  // fp32 node latents v^k (owned rows): every block's, or a ping-pong pair when checkpointing
  float* V(int k) const { return (float*)(ws + p.V) + (size_t)(p.lean || p.infer ? (k & 1) : k) * no * L; }
  float* AGG(int k) const { return (float*)(ws + p.AGG) + (size_t)(p.infer ? 0 : p.lean ? (k & 1) : k) * no * L; }
  // edge latents e^k: every block's, or the checkpoint slots plus one working slot
  void* ES(int k) const {
    const int slot = p.infer ? 0 : !p.lean ? k : (k % p.s == 0 ? k / p.s : p.nck);
    return (void*)(ws + p.ES + ts * (size_t)slot * ne * L);
  }
  int64_t v16_stride() const { return (no + nh) * L; }  // elements per block of the bf16 node copy
  void* V16(int k) const {
    return bf16 ? (void*)((uint16_t*)(ws + p.V16) + (size_t)(p.infer ? (k & 1) : k) * v16_stride()) : nullptr;
  }
};

// ---- forward, in three stages: encoders, one block at a time, decoder

mgn_status fwd_begin(mgn_model* m, const mgn_graph* g, const float* nf, const float* ef, const float* halo,
                     float* out, void* workspace, size_t ws_bytes, hipStream_t st, const char* fn) {
  const std::string f(fn);
  if (!m) return fail(nullptr, MGN_E_ARG, f + ": model is NULL");
  mgn_status s = check_graph_args(m, g);
  if (s) return s;
  if (!m->params_set) return fail(m, MGN_E_STATE, f + ": parameters were never set");
  if (!m->graph_ok || !same_graph(*g, m->vg))
    return fail(m, MGN_E_STATE, f + ": graph was not validated with mgn_graph_validate");
  const int64_t no = g->n_owned, nh = g->n_halo, ne = g->n_edges;
  if ((no > 0 && (!nf || !out)) || (ne > 0 && !ef)) return fail(m, MGN_E_ARG, f + ": input is NULL");
  if (nh > 0 && m->K > 0 && !halo) return fail(m, MGN_E_ARG, f + ": halo is NULL but n_halo > 0");
  if (!aligned(nf, 4) || !aligned(ef, 4) || !aligned(out, 4) || !aligned(halo, 16))
    return fail(m, MGN_E_ARG, f + ": misaligned pointer (features 4 bytes, halo 16 bytes)");
  if (!workspace || !aligned(workspace, 256))
    return fail(m, MGN_E_ARG, f + ": workspace NULL or not 256-byte aligned");
  const WsPlan p = make_plan(m, g);
  if (ws_bytes < p.total)
    return fail(m, MGN_E_NOMEM, f + ": workspace too small (need " + std::to_string(p.total) + " bytes)");
  // the step's buffers, kept for the later stages and the backward
  m->fwd_done = false;
  m->fwd_next = -1;
  m->bwd_active = false;
  m->g = *g;
  m->nf = nf;
  m->ef = ef;
  m->halo = halo;
  m->out = out;
  m->ws = (char*)workspace;
  m->plan = p;
  const Views b(m);
  const int L = m->L, K = m->K, D = m->D;
  const int te = edge_tile_rows(m->prec, L, D);
  hipError_t e;
  {
    Timed t_(m, MGN_T_OTHER, st);
    e = launch_erecv(g->row_ptr, no, (int32_t*)(b.ws + p.erecv), st);
    if (e == hipSuccess)
      e = launch_plan(g->row_ptr, no, 4 * te, 4 * te, (int32_t*)(b.ws + p.chunk), (int32_t*)(b.ws + p.unit_r),
                      (int32_t*)(b.ws + p.nunits), st);
  }
  if (e != hipSuccess) return hip_fail(m, e, (f + " plan").c_str());
  RowsFwdArgs ra{};
  ra.eps = m->cfg.ln_eps;
  // EncNode: v^0 for owned nodes
  ra.mlp = dev_mlp(m, m->enc_node());
  ra.rows = no;
  ra.fin = m->cfg.node_in;
  ra.in0 = nf;
  ra.out = b.V(0);
  ra.out16 = b.V16(0);
  {
    Timed t_(m, MGN_T_ENCODE, st);
    e = launch_rows_fwd(m->prec, L, D, ENC_NODE, ra, st);
  }
  if (e != hipSuccess) return hip_fail(m, e, (f + " EncNode").c_str());
  if (K > 0) {
    ra.mlp = dev_mlp(m, m->enc_edge());
    ra.rows = ne;
    ra.fin = m->cfg.edge_in;
    ra.in0 = ef;
    ra.out = b.ES(0);
    ra.out16 = nullptr;
    {
      Timed t_(m, MGN_T_ENCODE, st);
      e = launch_rows_fwd(m->prec, L, D, ENC_EDGE, ra, st);
    }
    if (e != hipSuccess) return hip_fail(m, e, (f + " EncEdge").c_str());
  }
  m->fwd_next = 0;
  return MGN_OK;
}

// Block k = fwd_next: reads halo[k] (when it runs), v^k, e^k; writes v^{k+1}, e^{k+1}.
mgn_status fwd_block(mgn_model* m, hipStream_t st, const char* fn) {
  const std::string f(fn);
  if (!m) return fail(nullptr, MGN_E_ARG, f + ": model is NULL");
  if (m->fwd_next < 0 || m->fwd_next >= m->K) return fail(m, MGN_E_STATE, f + ": no forward block is pending");
  const int k = m->fwd_next;
  m->fwd_next = -1;  // until the block is enqueued
  const Views b(m);
  const int L = m->L, K = m->K, D = m->D;
  const int64_t no = b.no, nh = b.nh;
  hipError_t e = hipSuccess;
  if (b.bf16 && nh > 0) {  // this block's halo rows of the bf16 node copy
    Timed t_(m, MGN_T_OTHER, st);
    e = launch_halo_bf16(m->halo + (size_t)k * nh * L, 1, nh, no, L, b.V16(k), b.v16_stride(), st);
    if (e != hipSuccess) return hip_fail(m, e, (f + " halo copy").c_str());
  }
  e = edge_forward_block(m, m->g, b.p, b.ws, m->halo, k, b.V(k), b.V16(k), b.ES(k), k + 1 < K ? b.ES(k + 1) : nullptr,
                         b.AGG(k), st);
  if (e != hipSuccess) return hip_fail(m, e, (f + " edge block").c_str());
  RowsFwdArgs na{};
  na.mlp = dev_mlp(m, m->node(k));
  na.rows = no;
  na.in0 = b.V(k);
  na.in1 = b.AGG(k);
  na.out = b.V(k + 1);
  na.out16 = b.V16(k + 1);
  na.in0_16 = b.V16(k);
  na.hid_out = (b.p.HID_NK && !b.p.lean) ? (void*)((uint16_t*)(b.ws + b.p.HID_NK) + (size_t)k * no * L) : nullptr;
  na.eps = m->cfg.ln_eps;
  {
    Timed t_(m, MGN_T_NODE_FWD, st);
    e = launch_rows_fwd(m->prec, L, D, NODE_BLOCK, na, st);
  }
  if (e != hipSuccess) return hip_fail(m, e, (f + " node block").c_str());
  m->fwd_next = k + 1;
  return MGN_OK;
}

mgn_status fwd_end(mgn_model* m, hipStream_t st, const char* fn) {
  const std::string f(fn);
  if (!m) return fail(nullptr, MGN_E_ARG, f + ": model is NULL");
  if (m->fwd_next != m->K) return fail(m, MGN_E_STATE, f + ": the forward's blocks have not all run");
  m->fwd_next = -1;
  const Views b(m);
  RowsFwdArgs da{};
  da.mlp = dev_mlp(m, m->dec());
  da.rows = b.no;
  da.in0 = b.V(m->K);
  da.out = m->out;
  da.fout = m->cfg.node_out;
  da.eps = m->cfg.ln_eps;
  hipError_t e;
  {
    Timed t_(m, MGN_T_DECODE, st);
    e = launch_rows_fwd(m->prec, m->L, m->D, DECODER, da, st);
  }
  if (e != hipSuccess) return hip_fail(m, e, (f + " DecNode").c_str());
  m->fwd_done = true;
  m->agg_last = m->plan.lean;
  return MGN_OK;
}

// ---- backward, in three stages: decoder, one block at a time (K-1 .. 0), encoders

#define CHK(what) \
  if (e != hipSuccess) return hip_fail(m, e, "mgn_backward " what);

struct Bwd {
  mgn_model* m;
  hipStream_t st;
  Views b;
  const WsPlan& p;
  char* ws;
  const mgn_graph* g;
  int64_t no, nh, ne;
  int L, K, D;
  size_t ts;
  float* DV[2];
  void* DE;  // dL/de in the storage type
  float *DAGG, *DZS, *VP;
  int32_t* erecv;
  void *DEL_N[3], *HID_N[2], *DEL_E[3], *HID_E[2];
  float* d_params;
  int accumulate;
  size_t nch;  // edge chunks of the backward

  Bwd(mgn_model* m_, hipStream_t s)
      : m(m_), st(s), b(m_), p(m_->plan), ws(m_->ws), g(&m_->g), no(b.no), nh(b.nh), ne(b.ne), L(m_->L), K(m_->K),
        D(m_->D), ts(b.ts), d_params(m_->d_params), accumulate(m_->accumulate) {
    DV[0] = (float*)(ws + p.DV[0]);
    DV[1] = (float*)(ws + p.DV[1]);
    DE = ws + p.DE;
    DAGG = (float*)(ws + p.DAGG);
    DZS = (float*)(ws + p.DZS);
    VP = (float*)(ws + p.VPART);
    erecv = (int32_t*)(ws + p.erecv);
    for (int j = 0; j < 3; ++j) DEL_N[j] = ws + p.DEL_N[j];
    for (int j = 0; j < 2; ++j) HID_N[j] = ws + p.HID_N[j];
    for (int j = 0; j < 3; ++j) DEL_E[j] = ws + p.DEL_E[j];
    for (int j = 0; j < 2; ++j) HID_E[j] = ws + p.HID_E[j];
    nch = p.cr.size() - 1;
  }

  RowsBwdArgs rows_args(const MlpL& ml, int64_t rows, void* const* del, void* const* hid) const {
    RowsBwdArgs a{};
    a.mlp = dev_mlp(m, ml);
    a.rows = rows;
    a.vpart = VP;
    a.nvec = ml.nvec;
    a.eps = m->cfg.ln_eps;
    for (int j = 0; j < 3; ++j) a.delta[j] = del[j];
    for (int j = 0; j < 2; ++j) a.hid[j] = hid[j];
    return a;
  }

  // weight gradients of the hidden / last Linears from the stored activations
  hipError_t dw_hidden(const MlpL& ml, int64_t R, void* const* del, void* const* hid, int ld_last, int acc) {
    for (int j = 1; j < D; ++j) {
      DwArgs a{};
      a.delta = del[j];
      a.ldd = (j == D - 1) ? ld_last : L;
      a.a_kind = 0;
      a.a0 = hid[j - 1];
      a.lda0 = L;
      a.R = R;
      hipError_t r = run_dw(m, ml.lin[j], a, d_params, acc, st);
      if (r != hipSuccess) return r;
    }
    return hipSuccess;
  }

  // DecNode: dL/dv^K into DV[0]
  mgn_status decoder(const float* d_out) {
    hipError_t e;
    const MlpL& ml = m->dec();
    RowsBwdArgs a = rows_args(ml, no, DEL_N, HID_N);
    a.in0 = b.V(K);
    a.dm = d_out;
    a.dx0 = DV[0];
    a.fout = m->cfg.node_out;
    {
      Timed t_(m, MGN_T_NODE_BWD, st);
      e = launch_rows_bwd(m->prec, L, D, DECODER, a, BWD_GRID, st);
    }
    CHK("decoder");
    e = run_vec(m, ml, d_params, accumulate, st);
    CHK("decoder vec");
    DwArgs w{};
    w.delta = DEL_N[0];
    w.ldd = L;
    w.a_kind = 1;
    w.a0 = b.V(K);
    w.lda0 = L;
    w.R = no;
    e = run_dw(m, ml.lin[0], w, d_params, accumulate, st);
    CHK("decoder dW");
    e = dw_hidden(ml, no, DEL_N, HID_N, 16, accumulate);
    CHK("decoder dW");
    return MGN_OK;
  }

  // Block k: DV[a_] holds dL/dv^{k+1} (owned rows); writes dL/dv^k into
  // DV[1 - a_] and dL/dhalo[k] into d_halo_k (when not null).
  mgn_status block(int k, int a_, float* d_halo_k) {
    hipError_t e = hipSuccess;
    const int b_ = 1 - a_;
    const float* Hk = nh > 0 ? m->halo + (size_t)k * nh * L : nullptr;
    if (p.lean) {
      // e^k: the edge forwards of blocks b0 .. k-1 from the checkpoint e^{b0}
      // (their aggregates into block k-1's slot: the last one is agg^{k-1},
      // which block k-1's backward then reads).  agg^k is in block k's slot
      // when block k+1's recompute ended with block k; otherwise block k's
      // forward runs once more for it.
      const int b0 = k - k % p.s;
      for (int j = b0; j < k; ++j) {
        e = edge_forward_block(m, *g, p, ws, m->halo, j, b.V(j), b.V16(j), b.ES(j), b.ES(j + 1), b.AGG(k - 1), st);
        CHK("edge-stream recompute");
      }
      // the last block's aggregate is still where the forward left it
      // unless an earlier backward has run since
      const bool have_agg = k + 1 < K ? (k + 1) % p.s != 0 : m->agg_last;
      m->agg_last = false;
      if (!have_agg) {
        e = edge_forward_block(m, *g, p, ws, m->halo, k, b.V(k), b.V16(k), b.ES(k), nullptr, b.AGG(k), st);
        CHK("aggregate recompute");
      } else if ((edge_rs(m->prec, L, D) || edge_rsb(m->prec, L, D)) && no > 0) {
        // block k's node projections for its edge backward (the slot holds block k-1's)
        Timed t_(m, MGN_T_NODE_PROJ, st);
        e = launch_node_proj(L, b.V16(k), no + nh, dev_mlp(m, m->edge(k)).lin[0], proj_block(p, ws, k, no + nh, L), st);
        CHK("projections");
      }
    }
    {
      const MlpL& ml = m->node(k);
      RowsBwdArgs a = rows_args(ml, no, DEL_N, HID_N);
      a.in0 = p.lean ? nullptr : b.V(k);
      a.in0_16 = p.lean ? b.V16(k) : nullptr;  // the bf16 copy is the product operand either way
      a.in1 = b.AGG(k);
      void* hidk[2] = {HID_N[0], HID_N[1]};
      if (p.HID_NK) {  // the forward's ReLU output of this block
        uint16_t* hk = (uint16_t*)(ws + p.HID_NK) + (p.lean ? 0 : (size_t)k * no * L);
        if (p.lean && no > 0) {  // recomputed from the block's inputs by the same kernel
          RowsFwdArgs ra{};
          ra.mlp = a.mlp;
          ra.rows = no;
          ra.in1 = b.AGG(k);
          ra.in0_16 = b.V16(k);
          ra.hid_out = hk;
          ra.eps = m->cfg.ln_eps;
          Timed t_(m, MGN_T_NODE_BWD, st);
          e = launch_rows_fwd(m->prec, L, D, NODE_BLOCK, ra, st);
          CHK("node ReLU output recompute");
        }
        a.hid_in = hk;
        hidk[0] = hk;
      }
      a.dm = DV[a_];
      a.dx0 = DV[b_];
      a.dx1 = DAGG;
      {
        Timed t_(m, MGN_T_NODE_BWD, st);
        e = launch_rows_bwd(m->prec, L, D, NODE_BLOCK, a, BWD_GRID, st);
      }
      CHK("node block");
      e = run_vec(m, ml, d_params, accumulate, st, rows_bwd_grid(m->prec, L, D, NODE_BLOCK, BWD_GRID));
      CHK("node vec");
      // first Linear, input [v | agg]: one weight gradient per column block
      // (each a plain row-major operand, so the register-resident kernels
      // take them at l = 128); fp32 rows enter bf16 products rounded
      DwArgs w{};
      w.delta = DEL_N[0];
      w.ldd = L;
      w.lda0 = L;
      w.R = no;
      const bool st_v = m->prec == F32 || !p.lean;  // v in the storage type (fp32 V) or bf16 copy
      w.a_kind = (m->prec == BF16 && !p.lean) ? 1 : 0;
      w.a0 = st_v ? (const void*)b.V(k) : b.V16(k);
      e = run_dw(m, ml.lin[0], w, d_params, accumulate, st, 0, L);
      CHK("node dW (v block)");
      w.a_kind = m->prec == BF16 ? 1 : 0;
      w.a0 = b.AGG(k);
      e = run_dw(m, ml.lin[0], w, d_params, accumulate, st, L, L);
      CHK("node dW (agg block)");
      e = dw_hidden(ml, no, DEL_N, hidk, L, accumulate);
      CHK("node dW");
    }
    {
      const MlpL& ml = m->edge(k);
      EdgeBwdArgs a{};
      a.mlp = dev_mlp(m, ml);
      a.row_ptr = g->row_ptr;
      a.send = g->send;
      a.erecv = erecv;
      a.unit_r = (int32_t*)(ws + p.unit_r);
      a.n_units = (int32_t*)(ws + p.nunits);
      a.V = b.V(k);
      a.H = Hk;
      a.V16 = b.V16(k);
      a.n_owned = no;
      a.Ein = b.ES(k);
      a.de_next = (k == K - 1) ? nullptr : DE;  // dL/de is updated in place
      a.dagg = DAGG;
      a.de_out = DE;
      const bool rs = edge_rs(m->prec, L, D);
      // the forward's projections of block k (or those of the aggregate
      // recompute; with the l = 256 row-split forward the checkpointed plan's
      // recompute of the first layer uses them too)
      // the forward's first-Linear ReLU output of this block (stash-all
      // streaming path, or a stashed row-split block): not recomputed, and
      // the layer-2 weight gradient reads it in place
      void* h1 = h1_slot(p, ws, k, ts * (size_t)ne * L);
      // (a stashed row-split block's projection slot is shared and not read)
      a.proj = ((rs && !h1) || (p.lean && edge_rsb(m->prec, L, D))) ? proj_block(p, ws, k, no + nh, L) : nullptr;
      a.hid_in = h1;
      for (int j = 0; j < 3; ++j) a.delta[j] = DEL_E[j];
      for (int j = 0; j < 2; ++j) a.hid[j] = HID_E[j];
      a.vpart = VP;
      a.nvec = ml.nvec;
      a.eps = m->cfg.ln_eps;
      for (size_t c = 0; c < nch; ++c) {
        // one receiver chunk: its per-edge gradients are stored from edge ce[c]
        const int acc = accumulate || c > 0;
        const int64_t e0 = p.ce[c], rows = p.ce[c + 1] - p.ce[c];
        a.r_lo = p.cr[c];
        a.r_hi = p.cr[c + 1];
        a.e_base = e0;
        {
          Timed t_(m, MGN_T_EDGE_BWD, st);
          e = launch_edge_bwd(m->prec, L, D, a, BWD_GRID, st);
        }
        CHK("edge block");
        e = run_vec(m, ml, d_params, acc, st, edge_bwd_grid(m->prec, L, D, BWD_GRID));
        CHK("edge vec");
        void* hid_c[2] = {h1 ? (void*)((char*)h1 + ts * (size_t)e0 * L) : HID_E[0], HID_E[1]};
        e = dw_hidden(ml, rows, DEL_E, hid_c, L, acc);
        CHK("edge dW");
        // first Linear's weight gradient, e block: e rows of the chunk
        DwArgs w{};
        w.delta = DEL_E[0];
        w.ldd = L;
        w.a_kind = 0;
        w.a0 = (const char*)b.ES(k) + ts * (size_t)e0 * L;
        w.lda0 = L;
        w.R = rows;
        e = run_dw(m, ml.lin[0], w, d_params, acc, st, 0, L);
        CHK("edge dW (e block)");
        if (nch > 1) {
          // per-sender sums of dz_0, chunk by chunk in ascending edge order:
          // zero once, then each chunk adds to the senders of its edges only
          Timed t_(m, MGN_T_INPUT_GRAD, st);
          int32_t* sr = (int32_t*)(ws + p.SRANGE);
          if (c == 0) e = launch_zero(DZS, (no + nh) * (int64_t)L, st);
          if (e == hipSuccess) e = launch_sender_range(g->send, e0, e0 + rows, sr, st);
          if (e == hipSuccess)
            e = launch_sender_sums(m->prec, L, g->trow_ptr, g->tedge, DEL_E[0], e0, e0 + rows, no + nh, DZS, 0, sr,
                                   st);
          CHK("sender sums");
        }
      }
      InGradArgs ig{};
      ig.w1 = a.mlp.lin[0];
      ig.trow = g->trow_ptr;
      ig.tedge = g->tedge;
      ig.dz = DEL_E[0];
      ig.dzr = DAGG;
      ig.dv = DV[b_];
      ig.dh = d_halo_k;
      ig.dzs = DZS;
      ig.dzs_ready = nch > 1;
      ig.n_local = no + nh;
      ig.n_owned = no;
      {
        Timed t_(m, MGN_T_INPUT_GRAD, st);
        e = launch_input_grad(m->prec, L, ig, st);
      }
      CHK("node input gradient");
      // the first Linear's sender / receiver weight-gradient blocks as sums
      // over nodes of (per-node sum of dz_0) times the node's v (the same
      // sums as over edges, reassociated)
      for (int side = 0; side < 2; ++side) {  // sender block, then receiver block
        DwArgs wn{};
        wn.delta = side == 0 ? (const void*)DZS : (const void*)DAGG;
        wn.d_kind = 1;
        wn.ldd = L;
        wn.lda0 = L;
        wn.R = side == 0 ? no + nh : no;
        if (m->prec == BF16) {
          wn.a_kind = 0;
          wn.a0 = b.V16(k);
        } else {
          wn.a_kind = 4;
          wn.a0 = b.V(k);
          wn.a2 = Hk;
          wn.n_owned = no;
        }
        e = run_dw(m, ml.lin[0], wn, d_params, accumulate, st, (1 + side) * L, L);
        CHK("edge dW (node blocks)");
      }
    }
    return MGN_OK;
  }

  // EncNode and EncEdge from dL/dv^0 (DV[a_]) and dL/de^0 (DE)
  mgn_status encoders(int a_) {
    hipError_t e = hipSuccess;
    {
      const MlpL& ml = m->enc_node();
      RowsBwdArgs a = rows_args(ml, no, DEL_N, HID_N);
      a.in0 = m->nf;
      a.fin = m->cfg.node_in;
      a.dm = DV[a_];
      {
        Timed t_(m, MGN_T_NODE_BWD, st);
        e = launch_rows_bwd(m->prec, L, D, ENC_NODE, a, BWD_GRID, st);
      }
      CHK("EncNode");
      e = run_vec(m, ml, d_params, accumulate, st, rows_bwd_grid(m->prec, L, D, ENC_NODE, BWD_GRID));
      CHK("EncNode vec");
      DwArgs w{};
      w.delta = DEL_N[0];
      w.ldd = L;
      w.a_kind = 1;
      w.a0 = m->nf;
      w.lda0 = m->cfg.node_in;
      w.R = no;
      e = run_dw(m, ml.lin[0], w, d_params, accumulate, st);
      CHK("EncNode dW");
      e = dw_hidden(ml, no, DEL_N, HID_N, L, accumulate);
      CHK("EncNode dW");
    }
    const MlpL& ml = m->enc_edge();
    if (K > 0 && ne > 0) {
      // over the same edge chunks as the blocks (per-edge gradients stored per chunk)
      for (size_t c = 0; c < nch; ++c) {
        const int acc = accumulate || c > 0;
        const int64_t e0 = p.ce[c], rows = p.ce[c + 1] - p.ce[c];
        RowsBwdArgs a = rows_args(ml, rows, DEL_E, HID_E);
        a.in0 = m->ef + (size_t)e0 * m->cfg.edge_in;
        a.fin = m->cfg.edge_in;
        // dL/de^0 (block 0 wrote it in plain column order, in the storage type)
        if (m->prec == BF16) a.dm16 = (const uint16_t*)DE + (size_t)e0 * L;
        else a.dm = (const float*)DE + (size_t)e0 * L;
        // narrow features: the kernel forms the first Linear's weight
        // gradient itself (per-wave partials) instead of storing dz_0
        const int w1s = rows > 0 ? rows_rt_w1_parts(m->prec, L, D, ENC_EDGE, a.fin) : 0;
        if (w1s) a.w1_part = (float*)(ws + p.PART);
        {
          Timed t_(m, MGN_T_NODE_BWD, st);
          e = launch_rows_bwd(m->prec, L, D, ENC_EDGE, a, BWD_GRID, st);
        }
        CHK("EncEdge");
        e = run_vec(m, ml, d_params, acc, st, rows_bwd_grid(m->prec, L, D, ENC_EDGE, BWD_GRID));
        CHK("EncEdge vec");
        if (w1s) {
          Timed t_(m, MGN_T_WEIGHT_GRAD, st);
          e = launch_dw_reduce(a.w1_part, w1s, L, a.fin, d_params + ml.lin[0].w, a.fin, acc, st);
        } else {
          DwArgs w{};
          w.delta = DEL_E[0];
          w.ldd = L;
          w.a_kind = 1;
          w.a0 = a.in0;
          w.lda0 = m->cfg.edge_in;
          w.R = rows;
          e = run_dw(m, ml.lin[0], w, d_params, acc, st);
        }
        CHK("EncEdge dW");
        e = dw_hidden(ml, rows, DEL_E, HID_E, L, acc);
        CHK("EncEdge dW");
      }
    } else if (!accumulate) {
      // no edges reach the output: the edge encoder's gradient is zero
      const int64_t b0 = ml.lin[0].w;
      const int64_t end = ml.beta + ml.lin[D - 1].out;
      e = launch_zero(d_params + b0, end - b0, st);
      CHK("EncEdge zero");
    }
    return MGN_OK;
  }
};

#undef CHK

mgn_status bwd_begin(mgn_model* m, const float* d_out, float* d_params, int accumulate, float* d_halo,
                     hipStream_t st, const char* fn) {
  const std::string f(fn);
  if (!m) return fail(nullptr, MGN_E_ARG, f + ": model is NULL");
  if (!m->fwd_done) return fail(m, MGN_E_STATE, f + ": no forward pass to differentiate");
  if (m->plan.infer) return fail(m, MGN_E_STATE, f + ": the forward pass ran in inference mode");
  if (!m->graph_ok || !same_graph(m->g, m->vg))
    return fail(m, MGN_E_STATE, f + ": the graph changed since the forward pass");
  if (!d_params || (m->g.n_owned > 0 && !d_out)) return fail(m, MGN_E_ARG, f + ": NULL argument");
  if (!aligned(d_out, 4) || !aligned(d_params, 4) || !aligned(d_halo, 16))
    return fail(m, MGN_E_ARG, f + ": misaligned pointer (d_halo 16 bytes)");
  m->bwd_active = false;
  m->d_params = d_params;
  m->accumulate = accumulate;
  m->d_halo = d_halo;
  Bwd w(m, st);
  mgn_status s = w.decoder(d_out);
  if (s) return s;
  m->bwd_active = true;
  m->bwd_next = m->K - 1;
  m->bwd_a = 0;
  return MGN_OK;
}

mgn_status bwd_block(mgn_model* m, hipStream_t st, const char* fn) {
  const std::string f(fn);
  if (!m) return fail(nullptr, MGN_E_ARG, f + ": model is NULL");
  if (!m->bwd_active || !m->fwd_done || m->bwd_next < 0)
    return fail(m, MGN_E_STATE, f + ": no backward block is pending");
  const int k = m->bwd_next;
  m->bwd_active = false;  // until the block is enqueued
  Bwd w(m, st);
  const int64_t nh = m->g.n_halo;
  mgn_status s = w.block(k, m->bwd_a, m->d_halo ? m->d_halo + (size_t)k * nh * m->L : nullptr);
  if (s) return s;
  m->bwd_a = 1 - m->bwd_a;
  m->bwd_next = k - 1;
  m->bwd_active = true;
  return MGN_OK;
}

mgn_status bwd_end(mgn_model* m, hipStream_t st, const char* fn) {
  const std::string f(fn);
  if (!m) return fail(nullptr, MGN_E_ARG, f + ": model is NULL");
  if (!m->bwd_active || !m->fwd_done || m->bwd_next != -1)
    return fail(m, MGN_E_STATE, f + ": the backward's blocks have not all run");
  m->bwd_active = false;
  Bwd w(m, st);
  return w.encoders(m->bwd_a);
}

}  // namespace

extern "C" {

mgn_status mgn_forward(mgn_model* m, const mgn_graph* g, const float* nf, const float* ef, const float* halo,
                       float* out, void* workspace, size_t ws_bytes, mgn_stream stream) {
  hipStream_t st = (hipStream_t)stream;
  mgn_status s = fwd_begin(m, g, nf, ef, halo, out, workspace, ws_bytes, st, "mgn_forward");
  for (int k = 0; s == MGN_OK && k < m->K; ++k) s = fwd_block(m, st, "mgn_forward");
  if (s == MGN_OK) s = fwd_end(m, st, "mgn_forward");
  return s;
}

mgn_status mgn_forward_begin(mgn_model* m, const mgn_graph* g, const float* nf, const float* ef, const float* halo,
                             float* out, void* workspace, size_t ws_bytes, mgn_stream stream) {
  return fwd_begin(m, g, nf, ef, halo, out, workspace, ws_bytes, (hipStream_t)stream, "mgn_forward_begin");
}

mgn_status mgn_forward_block(mgn_model* m, mgn_stream stream) {
  return fwd_block(m, (hipStream_t)stream, "mgn_forward_block");
}

mgn_status mgn_forward_end(mgn_model* m, mgn_stream stream) {
  return fwd_end(m, (hipStream_t)stream, "mgn_forward_end");
}

mgn_status mgn_backward(mgn_model* m, const float* d_out, float* d_params, int accumulate, float* d_halo,
                        mgn_stream stream) {
  hipStream_t st = (hipStream_t)stream;
  mgn_status s = bwd_begin(m, d_out, d_params, accumulate, d_halo, st, "mgn_backward");
  for (int k = 0; s == MGN_OK && k < m->K; ++k) s = bwd_block(m, st, "mgn_backward");
  if (s == MGN_OK) s = bwd_end(m, st, "mgn_backward");
  return s;
}

mgn_status mgn_backward_begin(mgn_model* m, const float* d_out, float* d_params, int accumulate, float* d_halo,
                              mgn_stream stream) {
  return bwd_begin(m, d_out, d_params, accumulate, d_halo, (hipStream_t)stream, "mgn_backward_begin");
}

mgn_status mgn_backward_block(mgn_model* m, mgn_stream stream) {
  return bwd_block(m, (hipStream_t)stream, "mgn_backward_block");
}

mgn_status mgn_backward_end(mgn_model* m, mgn_stream stream) {
  return bwd_end(m, (hipStream_t)stream, "mgn_backward_end");
}

mgn_status mgn_halo_masks(const int32_t* l2g_p, int64_t n_owned_p, int64_t n_halo_p, const int32_t* part,
                          int64_t n_nodes, const int32_t* l2g_q, int64_t n_owned_q, int32_t q, int32_t* recv_idx,
                          int32_t* send_rows, int64_t* count) {
  return halo_masks(l2g_p, n_owned_p, n_halo_p, part, n_nodes, l2g_q, n_owned_q, q, recv_idx, send_rows, count,
                    g_err);
}

mgn_status mgn_copy_latents(const mgn_model* owner, const int32_t* send_rows, const int32_t* recv_idx, int64_t n,
                            float* halo_k, int64_t n_halo, mgn_stream stream) {
  mgn_model* m = const_cast<mgn_model*>(owner);
  if (!m) return fail(nullptr, MGN_E_ARG, "mgn_copy_latents: model is NULL");
  if (n < 0 || n_halo < 0) return fail(m, MGN_E_ARG, "mgn_copy_latents: negative size");
  if (n == 0) return MGN_OK;
  if (!send_rows || !recv_idx || !halo_k) return fail(m, MGN_E_ARG, "mgn_copy_latents: NULL argument");
  if (!aligned(send_rows, 4) || !aligned(recv_idx, 4) || !aligned(halo_k, 16))
    return fail(m, MGN_E_ARG, "mgn_copy_latents: misaligned pointer (halo_k 16 bytes)");
  int j;
  if (m->fwd_next >= 0)
    j = m->fwd_next;
  else if (m->fwd_done)
    j = m->K;
  else
    return fail(m, MGN_E_STATE, "mgn_copy_latents: the owner has no forward pass in progress or done");
  const Views b(m);
  Timed t_(m, MGN_T_EXCHANGE, (hipStream_t)stream);
  hipError_t e = launch_rows_copy(b.V(j), b.no, send_rows, recv_idx, n, m->L, halo_k, n_halo, 0, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(m, e, "mgn_copy_latents");
  return MGN_OK;
}

mgn_status mgn_add_latent_grads(mgn_model* owner, const float* d_halo_k, int64_t n_halo, const int32_t* recv_idx,
                                const int32_t* send_rows, int64_t n, mgn_stream stream) {
  mgn_model* m = owner;
  if (!m) return fail(nullptr, MGN_E_ARG, "mgn_add_latent_grads: model is NULL");
  if (n < 0 || n_halo < 0) return fail(m, MGN_E_ARG, "mgn_add_latent_grads: negative size");
  if (!m->bwd_active || !m->fwd_done)
    return fail(m, MGN_E_STATE, "mgn_add_latent_grads: the owner has no backward pass in progress");
  if (n == 0) return MGN_OK;
  if (!send_rows || !recv_idx || !d_halo_k) return fail(m, MGN_E_ARG, "mgn_add_latent_grads: NULL argument");
  if (!aligned(send_rows, 4) || !aligned(recv_idx, 4) || !aligned(d_halo_k, 16))
    return fail(m, MGN_E_ARG, "mgn_add_latent_grads: misaligned pointer (d_halo_k 16 bytes)");
  const Views b(m);
  float* dv = (float*)(b.ws + b.p.DV[m->bwd_a]);
  Timed t_(m, MGN_T_EXCHANGE, (hipStream_t)stream);
  hipError_t e =
      launch_rows_copy(d_halo_k, n_halo, recv_idx, send_rows, n, m->L, dv, b.no, 1, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(m, e, "mgn_add_latent_grads");
  return MGN_OK;
}

}  // extern "C"

// Lockstep step of several parts on one device (one stream): the staged
// calls in Algorithm 1's order with the halo exchange between the blocks.
namespace {
mgn_status check_links(int32_t n_parts, mgn_model* const* models, const mgn_halo_link* links, int32_t n_links,
                       float* const* bufs, const char* fn) {
  const std::string f(fn);
  if (n_parts < 1 || !models || n_links < 0 || (n_links > 0 && !links))
    return fail(nullptr, MGN_E_ARG, f + ": bad part or link counts");
  for (int32_t p = 0; p < n_parts; ++p)
    if (!models[p]) return fail(nullptr, MGN_E_ARG, f + ": model is NULL");
  for (int32_t i = 0; i < n_links; ++i) {
    const mgn_halo_link& k = links[i];
    if (k.part < 0 || k.part >= n_parts || k.owner < 0 || k.owner >= n_parts || k.part == k.owner || k.n < 0)
      return fail(nullptr, MGN_E_ARG, f + ": link " + std::to_string(i) + " names a bad part");
    if (models[k.part]->L != models[k.owner]->L || models[k.part]->K != models[k.owner]->K)
      return fail(nullptr, MGN_E_ARG, f + ": linked parts have different latent sizes or block counts");
    if (k.n > 0 && (!k.recv_idx || !k.send_rows || !bufs || !bufs[k.part]))
      return fail(nullptr, MGN_E_ARG, f + ": link " + std::to_string(i) + " without index arrays or buffer");
  }
  return MGN_OK;
}
}  // namespace

extern "C" {

mgn_status mgn_lockstep_forward(int32_t n_parts, mgn_model* const* models, const mgn_graph* graphs,
                                const float* const* node_feat, const float* const* edge_feat, float* const* halo,
                                float* const* out, void* const* workspace, const size_t* ws_bytes,
                                const mgn_halo_link* links, int32_t n_links, mgn_stream stream) {
  mgn_status s = check_links(n_parts, models, links, n_links, halo, "mgn_lockstep_forward");
  if (s) return s;
  if (!graphs || !node_feat || !edge_feat || !out || !workspace || !ws_bytes)
    return fail(nullptr, MGN_E_ARG, "mgn_lockstep_forward: NULL array");
  hipStream_t st = (hipStream_t)stream;
  for (int32_t p = 0; p < n_parts; ++p) {
    s = fwd_begin(models[p], &graphs[p], node_feat[p], edge_feat[p], halo ? halo[p] : nullptr, out[p], workspace[p],
                  ws_bytes[p], st, "mgn_lockstep_forward");
    if (s) return s;
  }
  const int K = models[0]->K;
  for (int k = 0; k < K; ++k) {
    for (int32_t i = 0; i < n_links; ++i) {
      const mgn_halo_link& ln = links[i];
      if (ln.n == 0) continue;
      const int64_t nh = graphs[ln.part].n_halo;
      s = mgn_copy_latents(models[ln.owner], ln.send_rows, ln.recv_idx, ln.n,
                           halo[ln.part] + (size_t)k * nh * models[ln.part]->L, nh, stream);
      if (s) return fail(nullptr, s, std::string("mgn_lockstep_forward: ") + mgn_last_error(models[ln.owner]));
    }
    for (int32_t p = 0; p < n_parts; ++p) {
      s = fwd_block(models[p], st, "mgn_lockstep_forward");
      if (s) return s;
    }
  }
  for (int32_t p = 0; p < n_parts; ++p) {
    s = fwd_end(models[p], st, "mgn_lockstep_forward");
    if (s) return s;
  }
  return MGN_OK;
}

mgn_status mgn_lockstep_backward(int32_t n_parts, mgn_model* const* models, const float* const* d_out,
                                 float* d_params, int accumulate, float* const* d_halo, const mgn_halo_link* links,
                                 int32_t n_links, mgn_stream stream) {
  mgn_status s = check_links(n_parts, models, links, n_links, d_halo, "mgn_lockstep_backward");
  if (s) return s;
  if (!d_out) return fail(nullptr, MGN_E_ARG, "mgn_lockstep_backward: NULL array");
  hipStream_t st = (hipStream_t)stream;
  // one gradient buffer: the first part writes (or adds, accumulate), the others add, in part order
  for (int32_t p = 0; p < n_parts; ++p) {
    s = bwd_begin(models[p], d_out[p], d_params, accumulate || p > 0, d_halo ? d_halo[p] : nullptr, st,
                  "mgn_lockstep_backward");
    if (s) return s;
  }
  const int K = models[0]->K;
  for (int k = K - 1; k >= 0; --k) {
    for (int32_t p = 0; p < n_parts; ++p) {
      s = bwd_block(models[p], st, "mgn_lockstep_backward");
      if (s) return s;
    }
    for (int32_t i = 0; i < n_links; ++i) {
      const mgn_halo_link& ln = links[i];
      if (ln.n == 0) continue;
      mgn_model* mp = models[ln.part];
      const int64_t nh = mp->g.n_halo;
      s = mgn_add_latent_grads(models[ln.owner], d_halo[ln.part] + (size_t)k * nh * mp->L, nh, ln.recv_idx,
                               ln.send_rows, ln.n, stream);
      if (s) return fail(nullptr, s, std::string("mgn_lockstep_backward: ") + mgn_last_error(models[ln.owner]));
    }
  }
  for (int32_t p = 0; p < n_parts; ++p) {
    s = bwd_end(models[p], st, "mgn_lockstep_backward");
    if (s) return s;
  }
  return MGN_OK;
}

}  // extern "C"

extern "C" mgn_status mgn_mse_grad(const float* out, const float* target, const uint8_t* mask, int64_t n, int32_t d,
                                   float* loss, float* d_out, mgn_stream stream) {
  if (n < 0 || d < 1) return fail(nullptr, MGN_E_ARG, "mgn_mse_grad: bad sizes");
  if (!loss || (n > 0 && (!out || !target || !d_out))) return fail(nullptr, MGN_E_ARG, "mgn_mse_grad: NULL argument");
  hipError_t e = launch_mse(out, target, mask, n, d, 0, loss, d_out, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(nullptr, e, "mgn_mse_grad");
  return MGN_OK;
}

extern "C" mgn_status mgn_mse_grad_global(const float* out, const float* target, const uint8_t* mask, int64_t n,
                                          int32_t d, int64_t global_rows, float* loss, float* d_out,
                                          mgn_stream stream) {
  if (n < 0 || d < 1 || global_rows < 1) return fail(nullptr, MGN_E_ARG, "mgn_mse_grad_global: bad sizes");
  if (!loss || (n > 0 && (!out || !target || !d_out)))
    return fail(nullptr, MGN_E_ARG, "mgn_mse_grad_global: NULL argument");
  hipError_t e = launch_mse(out, target, mask, n, d, global_rows, loss, d_out, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(nullptr, e, "mgn_mse_grad_global");
  return MGN_OK;
}

extern "C" mgn_status mgn_timing_enable(mgn_model* m, int enable) {
  if (!m) return fail(nullptr, MGN_E_ARG, "mgn_timing_enable: model is NULL");
  m->timing = enable != 0;
  if (m->timing) {
    m->ev_used = 0;
    m->ev_rec.clear();
  }
  return MGN_OK;
}

extern "C" mgn_status mgn_timing_read(mgn_model* m, int timer, double* ms_total, int64_t* launches) {
  if (!m) return fail(nullptr, MGN_E_ARG, "mgn_timing_read: model is NULL");
  if (timer < 0 || timer >= MGN_T_COUNT || !ms_total || !launches)
    return fail(m, MGN_E_ARG, "mgn_timing_read: bad argument");
  double t = 0;
  int64_t n = 0;
  for (const auto& r : m->ev_rec) {
    if (r.first != timer) continue;
    hipError_t e = hipEventSynchronize(m->ev_pool[r.second + 1]);
    float ms = 0;
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, m->ev_pool[r.second], m->ev_pool[r.second + 1]);
    if (e != hipSuccess) return hip_fail(m, e, "mgn_timing_read");
    t += ms;
    ++n;
  }
  *ms_total = t;
  *launches = n;
  return MGN_OK;
}

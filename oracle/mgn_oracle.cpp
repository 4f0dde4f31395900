// CPU oracle for the MeshGraphNets training step -- TEST INFRASTRUCTURE ONLY.
//
// Only the tests, the smoke check and the CPU-baseline leg of the benchmark
// load this.  It is written to be read against the paper (section "Model",
// section "Methodology", Algorithm 1), not to be fast: float64 throughout,
// one row at a time, sums in ascending index order.  OpenMP only splits
// independent rows; weight-gradient sums use a fixed row chunking, so results
// do not depend on the thread count.
#include "mgn_oracle.h"

#include <algorithm>
#include <cmath>
#include <cstring>
#include <numeric>
#include <vector>

#ifdef _OPENMP
#include <omp.h>
#endif

namespace {

// ---------------------------------------------------------------- layout ---
struct Linear {
  int64_t w, b;  // offsets of W[out][in] and b[out] in the flat vector
  int in, out;
};

struct Mlp {
  std::vector<Linear> lin;
  bool ln = false;
  int64_t gamma = 0, beta = 0;
  int64_t begin = 0, size = 0;  // contiguous range of this MLP's parameters
  int in = 0, out = 0;
};

struct Model {
  orc_cfg c;
  Mlp enc_node, enc_edge, dec;
  std::vector<Mlp> edge, node;
  int64_t total = 0;
};

Mlp make_mlp(const orc_cfg& c, int fin, int fout, bool ln, int64_t& off) {
  Mlp m;
  m.begin = off;
  m.in = fin;
  m.out = fout;
  int prev = fin;
  for (int j = 0; j < c.depth; ++j) {
    int nxt = (j == c.depth - 1) ? fout : c.latent;
    Linear L{off, off + (int64_t)nxt * prev, prev, nxt};
    off += (int64_t)nxt * prev + nxt;
    m.lin.push_back(L);
    prev = nxt;
  }
  m.ln = ln;
  if (ln) {
    m.gamma = off;
    m.beta = off + fout;
    off += 2 * (int64_t)fout;
  }
  m.size = off - m.begin;
  return m;
}

bool valid(const orc_cfg* c) {
  return c && c->latent > 0 && c->n_blocks >= 0 && c->depth >= 2 && c->node_in > 0 &&
         c->edge_in > 0 && c->node_out > 0 && c->ln_eps > 0;
}

Model make_model(const orc_cfg& c) {
  Model m;
  m.c = c;
  int64_t off = 0;
  const int l = c.latent;
  m.enc_node = make_mlp(c, c.node_in, l, true, off);
  m.enc_edge = make_mlp(c, c.edge_in, l, true, off);
  for (int k = 0; k < c.n_blocks; ++k) {
    m.edge.push_back(make_mlp(c, 3 * l, l, true, off));
    m.node.push_back(make_mlp(c, 2 * l, l, true, off));
  }
  m.dec = make_mlp(c, l, c.node_out, false, off);
  m.total = off;
  return m;
}

// bfloat16 rounding as a single-precision kernel performs it: x is first a
// binary32 value, then rounded to the nearest value with 8 significant bits
// (ties to even): add half an ulp of the bfloat16 (minus one when the kept
// last bit is even) to the binary32 pattern and clear the low 16 bits.
double round_bf16(double x) {
  const float f = (float)x;
  if (!std::isfinite(f)) return x;
  uint32_t u;
  std::memcpy(&u, &f, 4);
  u += 0x7fffu + ((u >> 16) & 1u);
  u &= 0xffff0000u;
  float r;
  std::memcpy(&r, &u, 4);
  return (double)r;
}

// Weights as the matrix products see them (rounded copies in bf16 mode).
struct Params {
  const double* P;   // exact: biases, LayerNorm parameters
  const double* W;   // weights used in products
  bool bf16;
  double r(double x) const { return bf16 ? round_bf16(x) : x; }
};

// ------------------------------------------------------------- one MLP row ---
// Everything the backward pass needs from the forward pass of one row.
struct Trace {
  std::vector<std::vector<double>> a;  // a[j]: input of Linear j
  std::vector<std::vector<double>> z;  // z[j]: output of Linear j (pre-activation)
  std::vector<double> xhat;            // normalised output (LayerNorm only)
  double rstd = 0;
};

// y = LN(W_D ReLU(... ReLU(W_1 x + b_1) ...) + b_D), LN only if m.ln.
void mlp_forward(const Mlp& m, const Params& Q, double eps, const double* x, double* y, Trace& t) {
  const double* P = Q.P;
  const int D = (int)m.lin.size();
  t.a.resize(D);
  t.z.resize(D);
  t.a[0].resize(m.in);
  for (int i = 0; i < m.in; ++i) t.a[0][i] = Q.r(x[i]);
  for (int j = 0; j < D; ++j) {
    const Linear& L = m.lin[j];
    t.z[j].assign(L.out, 0.0);
    for (int o = 0; o < L.out; ++o) {
      double s = P[L.b + o];
      const double* w = Q.W + L.w + (int64_t)o * L.in;
      for (int i = 0; i < L.in; ++i) s += w[i] * t.a[j][i];
      t.z[j][o] = s;
    }
    if (j + 1 < D) {
      t.a[j + 1].resize(L.out);
      for (int o = 0; o < L.out; ++o) t.a[j + 1][o] = Q.r(t.z[j][o] > 0 ? t.z[j][o] : 0.0);
    }
  }
  const std::vector<double>& last = t.z[D - 1];
  const int n = m.out;
  if (!m.ln) {
    for (int o = 0; o < n; ++o) y[o] = last[o];
    return;
  }
  double mu = 0;
  for (int o = 0; o < n; ++o) mu += last[o];
  mu /= n;
  double var = 0;
  for (int o = 0; o < n; ++o) var += (last[o] - mu) * (last[o] - mu);
  var /= n;
  t.rstd = 1.0 / std::sqrt(var + eps);
  t.xhat.resize(n);
  for (int o = 0; o < n; ++o) {
    t.xhat[o] = (last[o] - mu) * t.rstd;
    y[o] = P[m.gamma + o] * t.xhat[o] + P[m.beta + o];
  }
}

// Reverse mode through the row traced in t: given dy = dL/dy, add the
// parameter gradients into g (indexed like the flat vector, relative to
// m.begin) and write dx = dL/dx.
void mlp_backward(const Mlp& m, const Params& Q, const Trace& t, const double* dy, double* dx,
                  double* g) {
  const double* P = Q.P;
  const int D = (int)m.lin.size();
  const int n = m.out;
  std::vector<double> dz(dy, dy + n);
  if (m.ln) {
    std::vector<double> dxh(n);
    for (int o = 0; o < n; ++o) {
      g[m.gamma - m.begin + o] += dy[o] * t.xhat[o];
      g[m.beta - m.begin + o] += dy[o];
      dxh[o] = dy[o] * P[m.gamma + o];
    }
    double mean_d = 0, mean_dx = 0;
    for (int o = 0; o < n; ++o) {
      mean_d += dxh[o];
      mean_dx += dxh[o] * t.xhat[o];
    }
    mean_d /= n;
    mean_dx /= n;
    for (int o = 0; o < n; ++o) dz[o] = t.rstd * (dxh[o] - mean_d - t.xhat[o] * mean_dx);
  }
  for (int j = D - 1; j >= 0; --j) {
    const Linear& L = m.lin[j];
    std::vector<double> da(L.in, 0.0);
    for (int o = 0; o < L.out; ++o) {
      g[L.b - m.begin + o] += dz[o];
      const double d = Q.r(dz[o]);
      double* gw = g + (L.w - m.begin) + (int64_t)o * L.in;
      const double* w = Q.W + L.w + (int64_t)o * L.in;
      for (int i = 0; i < L.in; ++i) {
        gw[i] += d * t.a[j][i];
        da[i] += w[i] * d;
      }
    }
    if (j == 0) {
      for (int i = 0; i < L.in; ++i) dx[i] = da[i];
    } else {
      dz.assign(L.in, 0.0);
      for (int i = 0; i < L.in; ++i) dz[i] = t.z[j - 1][i] > 0 ? da[i] : 0.0;
    }
  }
}

// Fixed chunking of `rows` rows for parameter-gradient sums.
int64_t chunk_rows(int64_t rows) { return std::max<int64_t>(1024, (rows + 63) / 64); }

// Runs body(row, trace, partial_grad) over all rows, each chunk of rows with
// its own zeroed partial gradient, then adds the partials into grad in chunk
// order.  body may write per-row outputs only.
template <class Body>
void rows_with_grad(int64_t rows, const Mlp& m, double* grad, Body body) {
  if (rows <= 0) return;
  const int64_t cr = chunk_rows(rows);
  const int64_t nch = (rows + cr - 1) / cr;
  std::vector<double> part((size_t)(nch * m.size), 0.0);
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t ch = 0; ch < nch; ++ch) {
    Trace t;
    double* g = part.data() + ch * m.size;
    const int64_t r1 = std::min(rows, (ch + 1) * cr);
    for (int64_t r = ch * cr; r < r1; ++r) body(r, t, g);
  }
  if (grad)
    for (int64_t ch = 0; ch < nch; ++ch)
      for (int64_t i = 0; i < m.size; ++i) grad[m.begin + i] += part[ch * m.size + i];
}

// ----------------------------------------------------------- the network ---
struct Graph {
  int64_t n_owned, n_halo, n_edges;
  const int32_t* row_ptr;
  const int32_t* send;
  std::vector<int32_t> recv;  // receiver of each local edge, from row_ptr
};

// One message-passing block's edge half: m[e] and e_next[e] (section "Model":
// each block is its own MLP applied to the previous block's output).
void edge_messages(const Model& M, const Mlp& em, const Params& Q, const Graph& G, const double* v,
                   const double* e, double* msg, double* e_next) {
  const int l = M.c.latent;
#pragma omp parallel for schedule(static)
  for (int64_t ed = 0; ed < G.n_edges; ++ed) {
    Trace t;
    std::vector<double> x(3 * l);
    const int64_t s = G.send[ed], r = G.recv[ed];
    for (int i = 0; i < l; ++i) {
      x[i] = e[ed * l + i];
      x[l + i] = v[s * l + i];
      x[2 * l + i] = v[r * l + i];
    }
    mlp_forward(em, Q, M.c.ln_eps, x.data(), msg + ed * l, t);
    if (e_next)
      for (int i = 0; i < l; ++i) e_next[ed * l + i] = Q.r(e[ed * l + i] + msg[ed * l + i]);
  }
}

void aggregate(const Graph& G, const double* msg, int l, double* agg) {
  orc_scatter_sum(G.n_owned, G.row_ptr, msg, l, agg);
}

void node_update(const Model& M, const Mlp& nm, const Params& Q, const Graph& G, const double* v,
                 const double* agg, double* v_next) {
  const int l = M.c.latent;
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < G.n_owned; ++r) {
    Trace t;
    std::vector<double> x(2 * l), y(l);
    for (int i = 0; i < l; ++i) {
      x[i] = v[r * l + i];
      x[l + i] = agg[r * l + i];
    }
    mlp_forward(nm, Q, M.c.ln_eps, x.data(), y.data(), t);
    for (int i = 0; i < l; ++i) v_next[r * l + i] = v[r * l + i] + y[i];
  }
}

}  // namespace

extern "C" {

int64_t orc_param_count(const orc_cfg* c) {
  if (!valid(c)) return -1;
  return make_model(*c).total;
}

int orc_partition(const int32_t* key, int64_t n, int32_t nparts, int32_t* part) {
  if (n < 0 || nparts < 1 || (n > 0 && (!key || !part))) return -1;
  std::vector<int64_t> order(n);
  std::iota(order.begin(), order.end(), 0);
  std::sort(order.begin(), order.end(), [&](int64_t a, int64_t b) {
    return key[a] != key[b] ? key[a] < key[b] : a < b;
  });
  for (int64_t q = 0; q < n; ++q) part[order[q]] = (int32_t)(((int64_t)nparts * q) / n);
  return 0;
}

int orc_graph_sizes(const int32_t* send, const int32_t* recv, int64_t n_edges, const int32_t* part,
                    int64_t n_nodes, int32_t p, int64_t* sizes) {
  if (n_edges < 0 || n_nodes < 0 || !sizes || (n_edges > 0 && (!send || !recv)) ||
      (n_nodes > 0 && !part))
    return -1;
  int64_t owned = 0, local = 0;
  for (int64_t g = 0; g < n_nodes; ++g) owned += part[g] == p;
  std::vector<char> is_halo(n_nodes, 0);
  for (int64_t e = 0; e < n_edges; ++e) {
    if (send[e] < 0 || send[e] >= n_nodes || recv[e] < 0 || recv[e] >= n_nodes) return -1;
    if (part[recv[e]] != p) continue;
    ++local;
    if (part[send[e]] != p) is_halo[send[e]] = 1;
  }
  int64_t halo = 0;
  for (int64_t g = 0; g < n_nodes; ++g) halo += is_halo[g];
  sizes[0] = owned;
  sizes[1] = halo;
  sizes[2] = local;
  return 0;
}

int orc_graph_build(const int32_t* send, const int32_t* recv, int64_t n_edges, const int32_t* part,
                    int64_t n_nodes, int32_t p, int32_t* row_ptr, int32_t* send_local,
                    int32_t* eperm, int32_t* trow_ptr, int32_t* tedge, int32_t* l2g) {
  int64_t sz[3];
  if (orc_graph_sizes(send, recv, n_edges, part, n_nodes, p, sz)) return -1;
  const int64_t no = sz[0], nh = sz[1], ne = sz[2];
  // local ids: owned by ascending global id, then halo by ascending global id
  std::vector<int64_t> g2l(n_nodes, -1);
  int64_t next = 0;
  for (int64_t g = 0; g < n_nodes; ++g)
    if (part[g] == p) g2l[g] = next++;
  std::vector<char> is_halo(n_nodes, 0);
  for (int64_t e = 0; e < n_edges; ++e)
    if (part[recv[e]] == p && part[send[e]] != p) is_halo[send[e]] = 1;
  for (int64_t g = 0; g < n_nodes; ++g)
    if (is_halo[g]) g2l[g] = next++;
  for (int64_t g = 0; g < n_nodes; ++g)
    if (g2l[g] >= 0) l2g[g2l[g]] = (int32_t)g;
  // local edges sorted by (local receiver, local sender, global edge id)
  std::vector<int64_t> le;
  le.reserve(ne);
  for (int64_t e = 0; e < n_edges; ++e)
    if (part[recv[e]] == p) le.push_back(e);
  std::sort(le.begin(), le.end(), [&](int64_t a, int64_t b) {
    if (g2l[recv[a]] != g2l[recv[b]]) return g2l[recv[a]] < g2l[recv[b]];
    if (g2l[send[a]] != g2l[send[b]]) return g2l[send[a]] < g2l[send[b]];
    return a < b;
  });
  for (int64_t r = 0; r <= no; ++r) row_ptr[r] = 0;
  for (int64_t i = 0; i < ne; ++i) {
    eperm[i] = (int32_t)le[i];
    send_local[i] = (int32_t)g2l[send[le[i]]];
    row_ptr[g2l[recv[le[i]]] + 1] += 1;
  }
  for (int64_t r = 0; r < no; ++r) row_ptr[r + 1] += row_ptr[r];
  // transposed CSR: per local sender, its local edges in ascending order
  const int64_t nl = no + nh;
  for (int64_t n = 0; n <= nl; ++n) trow_ptr[n] = 0;
  for (int64_t i = 0; i < ne; ++i) trow_ptr[send_local[i] + 1] += 1;
  for (int64_t n = 0; n < nl; ++n) trow_ptr[n + 1] += trow_ptr[n];
  std::vector<int64_t> fill(trow_ptr, trow_ptr + nl);
  for (int64_t i = 0; i < ne; ++i) tedge[fill[send_local[i]]++] = (int32_t)i;
  return 0;
}

int orc_edge_features(const double* coords, const int32_t* send, const int32_t* recv,
                      int64_t n_edges, double h, double* out) {
  if (n_edges < 0 || h <= 0) return -1;
  for (int64_t e = 0; e < n_edges; ++e) {
    double d[3], nn = 0;
    for (int a = 0; a < 3; ++a) {
      d[a] = (coords[3 * (int64_t)send[e] + a] - coords[3 * (int64_t)recv[e] + a]) / h;
      nn += d[a] * d[a];
    }
    for (int a = 0; a < 3; ++a) out[4 * e + a] = d[a];
    out[4 * e + 3] = std::sqrt(nn);
  }
  return 0;
}

int orc_scatter_sum(int64_t n_owned, const int32_t* row_ptr, const double* m, int32_t width,
                    double* agg) {
  if (n_owned < 0 || width <= 0) return -1;
  for (int64_t r = 0; r < n_owned; ++r) {
    for (int i = 0; i < width; ++i) agg[r * width + i] = 0.0;
    for (int64_t e = row_ptr[r]; e < row_ptr[r + 1]; ++e)
      for (int i = 0; i < width; ++i) agg[r * width + i] += m[e * width + i];
  }
  return 0;
}

int orc_step(const orc_cfg* c, int64_t n_owned, int64_t n_halo, int64_t n_edges,
             const int32_t* row_ptr, const int32_t* send, const double* P, const double* node_feat,
             const double* edge_feat, const double* halo, const double* d_out, double* out,
             double* d_params, double* d_halo, double* v_all, double* e_all) {
  if (!valid(c) || n_owned < 0 || n_halo < 0 || n_edges < 0 || !P || !out || !row_ptr) return -1;
  if ((n_edges > 0 && (!send || !edge_feat)) || (n_owned > 0 && !node_feat)) return -1;
  if (n_halo > 0 && c->n_blocks > 0 && !halo) return -1;
  if (d_out && !d_params) return -1;
  const Model M = make_model(*c);
  const int l = c->latent, K = c->n_blocks;
  const int64_t nl = n_owned + n_halo;
  Graph G{n_owned, n_halo, n_edges, row_ptr, send, std::vector<int32_t>(n_edges)};
  if (row_ptr[0] != 0 || row_ptr[n_owned] != n_edges) return -1;
  for (int64_t r = 0; r < n_owned; ++r) {
    if (row_ptr[r + 1] < row_ptr[r]) return -1;
    for (int64_t e = row_ptr[r]; e < row_ptr[r + 1]; ++e) G.recv[e] = (int32_t)r;
  }
  for (int64_t e = 0; e < n_edges; ++e)
    if (send[e] < 0 || send[e] >= nl) return -1;

  // weights as the products see them
  std::vector<double> Wr;
  if (c->bf16) {
    Wr.resize(M.total);
    for (int64_t i = 0; i < M.total; ++i) Wr[i] = round_bf16(P[i]);
  }
  const Params Q{P, c->bf16 ? Wr.data() : P, c->bf16 != 0};

  // stash of every block's inputs: v[k] (owned + halo rows), e[k]
  std::vector<std::vector<double>> V(K + 1, std::vector<double>(nl * l, 0.0));
  std::vector<std::vector<double>> E(K + 1, std::vector<double>(n_edges * l, 0.0));

  // encoders (Algorithm 1: EncNode, EncEdge)
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < n_owned; ++r) {
    Trace t;
    mlp_forward(M.enc_node, Q, c->ln_eps, node_feat + r * c->node_in, V[0].data() + r * l, t);
  }
#pragma omp parallel for schedule(static)
  for (int64_t e = 0; e < n_edges; ++e) {
    Trace t;
    mlp_forward(M.enc_edge, Q, c->ln_eps, edge_feat + e * c->edge_in, E[0].data() + e * l, t);
    for (int i = 0; i < l; ++i) E[0][e * l + i] = Q.r(E[0][e * l + i]);
  }

  // processor: K blocks, halo rows of each block's input from halo[k]
  std::vector<double> msg(n_edges * l), agg(n_owned * l);
  for (int k = 0; k < K; ++k) {
    for (int64_t h = 0; h < n_halo; ++h)
      for (int i = 0; i < l; ++i) V[k][(n_owned + h) * l + i] = halo[((int64_t)k * n_halo + h) * l + i];
    edge_messages(M, M.edge[k], Q, G, V[k].data(), E[k].data(), msg.data(), E[k + 1].data());
    aggregate(G, msg.data(), l, agg.data());
    node_update(M, M.node[k], Q, G, V[k].data(), agg.data(), V[k + 1].data());
  }

  // decoder
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < n_owned; ++r) {
    Trace t;
    mlp_forward(M.dec, Q, c->ln_eps, V[K].data() + r * l, out + r * c->node_out, t);
  }
  if (v_all)
    for (int k = 0; k <= K; ++k) std::memcpy(v_all + (int64_t)k * nl * l, V[k].data(), nl * l * 8);
  if (e_all)
    for (int k = 0; k <= K; ++k)
      std::memcpy(e_all + (int64_t)k * n_edges * l, E[k].data(), n_edges * l * 8);
  if (!d_out) return 0;

  // ------------------------------------------------------------ backward
  std::fill(d_params, d_params + M.total, 0.0);
  if (d_halo) std::fill(d_halo, d_halo + (int64_t)K * n_halo * l, 0.0);
  std::vector<double> dv(n_owned * l, 0.0), dv_next(n_owned * l), de(n_edges * l, 0.0),
      de_next(n_edges * l), dagg(n_owned * l), dxs(n_edges * l), dxr(n_edges * l);
  rows_with_grad(n_owned, M.dec, d_params, [&](int64_t r, Trace& t, double* g) {
    std::vector<double> y(c->node_out);
    mlp_forward(M.dec, Q, c->ln_eps, V[K].data() + r * l, y.data(), t);
    mlp_backward(M.dec, Q, t, d_out + r * c->node_out, dv.data() + r * l, g);
  });
  for (int k = K - 1; k >= 0; --k) {
    // the block's messages and aggregates again, from its stashed inputs
    edge_messages(M, M.edge[k], Q, G, V[k].data(), E[k].data(), msg.data(), nullptr);
    aggregate(G, msg.data(), l, agg.data());
    // node half: v_next = v + LN(MLP([v | agg]))
    rows_with_grad(n_owned, M.node[k], d_params, [&](int64_t r, Trace& t, double* g) {
      std::vector<double> x(2 * l), y(l), dx(2 * l);
      for (int i = 0; i < l; ++i) {
        x[i] = V[k][r * l + i];
        x[l + i] = agg[r * l + i];
      }
      mlp_forward(M.node[k], Q, c->ln_eps, x.data(), y.data(), t);
      mlp_backward(M.node[k], Q, t, dv.data() + r * l, dx.data(), g);
      for (int i = 0; i < l; ++i) {
        dv_next[r * l + i] = dv[r * l + i] + dx[i];
        dagg[r * l + i] = dx[l + i];
      }
    });
    // edge half: e_next = e + m, agg_r = sum m, m = LN(MLP([e | v_s | v_r]))
    rows_with_grad(n_edges, M.edge[k], d_params, [&](int64_t ed, Trace& t, double* g) {
      std::vector<double> x(3 * l), y(l), dm(l), dx(3 * l);
      const int64_t s = G.send[ed], r = G.recv[ed];
      for (int i = 0; i < l; ++i) {
        x[i] = E[k][ed * l + i];
        x[l + i] = V[k][s * l + i];
        x[2 * l + i] = V[k][r * l + i];
        dm[i] = de[ed * l + i] + dagg[r * l + i];
      }
      mlp_forward(M.edge[k], Q, c->ln_eps, x.data(), y.data(), t);
      mlp_backward(M.edge[k], Q, t, dm.data(), dx.data(), g);
      for (int i = 0; i < l; ++i) {
        // e^k is stored in bf16 in mixed precision, and so is its gradient
        de_next[ed * l + i] = Q.r(de[ed * l + i] + dx[i]);
        dxs[ed * l + i] = dx[l + i];
        dxr[ed * l + i] = dx[2 * l + i];
      }
    });
    // node gradients from the edges, ascending edge order
    for (int64_t ed = 0; ed < n_edges; ++ed) {
      const int64_t s = G.send[ed], r = G.recv[ed];
      for (int i = 0; i < l; ++i) dv_next[r * l + i] += dxr[ed * l + i];
      if (s < n_owned) {
        for (int i = 0; i < l; ++i) dv_next[s * l + i] += dxs[ed * l + i];
      } else if (d_halo) {
        double* dh = d_halo + ((int64_t)k * n_halo + (s - n_owned)) * l;
        for (int i = 0; i < l; ++i) dh[i] += dxs[ed * l + i];
      }
    }
    dv.swap(dv_next);
    de.swap(de_next);
  }
  // encoders
  rows_with_grad(n_owned, M.enc_node, d_params, [&](int64_t r, Trace& t, double* g) {
    std::vector<double> y(l), dx(c->node_in);
    mlp_forward(M.enc_node, Q, c->ln_eps, node_feat + r * c->node_in, y.data(), t);
    mlp_backward(M.enc_node, Q, t, dv.data() + r * l, dx.data(), g);
  });
  rows_with_grad(n_edges, M.enc_edge, d_params, [&](int64_t ed, Trace& t, double* g) {
    std::vector<double> y(l), dx(c->edge_in);
    mlp_forward(M.enc_edge, Q, c->ln_eps, edge_feat + ed * c->edge_in, y.data(), t);
    mlp_backward(M.enc_edge, Q, t, de.data() + ed * l, dx.data(), g);
  });
  return 0;
}

int orc_mse_grad(const double* out, const double* target, const uint8_t* mask, int64_t n, int32_t d,
                 double* loss, double* d_out) {
  return orc_mse_grad_global(out, target, mask, n, d, 0, loss, d_out);
}

// One part's share of the global mean over global_rows masked rows of all
// parts (Algorithm 1's loss all-reduce); global_rows = 0: this part's own rows.
int orc_mse_grad_global(const double* out, const double* target, const uint8_t* mask, int64_t n, int32_t d,
                        int64_t global_rows, double* loss, double* d_out) {
  if (n < 0 || d <= 0 || !loss || global_rows < 0) return -1;
  int64_t cnt = 0;
  for (int64_t i = 0; i < n; ++i) cnt += mask ? (mask[i] != 0) : 1;
  if (global_rows > 0) cnt = global_rows;
  const double denom = (double)cnt * d;
  double L = 0;
  for (int64_t i = 0; i < n; ++i) {
    const bool on = mask ? mask[i] != 0 : true;
    for (int j = 0; j < d; ++j) {
      const double diff = out[i * d + j] - target[i * d + j];
      if (on) L += diff * diff;
      if (d_out) d_out[i * d + j] = (on && cnt > 0) ? 2.0 * diff / denom : 0.0;
    }
  }
  *loss = cnt > 0 ? L / denom : 0.0;
  return 0;
}

// Algorithm 1's parameter update after the accumulated gradient:
// theta <- theta - eta * grad, element by element.
int orc_sgd_step(double* params, const double* grad, int64_t n, double lr) {
  if (n < 0 || (n > 0 && (!params || !grad))) return -1;
  for (int64_t i = 0; i < n; ++i) params[i] = params[i] - lr * grad[i];
  return 0;
}

// Next-step prediction (section "Model"): the network's output is the
// increment of the flow quantities, q_{t+1} = p_t + q_t, which sit in node
// feature columns col0 .. col0 + node_out - 1.
int orc_rollout_update(double* node_feat, int64_t n, int32_t node_in, const double* out, int32_t node_out,
                       int32_t col0) {
  if (n < 0 || col0 < 0 || node_out < 1 || col0 + node_out > node_in || (n > 0 && (!node_feat || !out))) return -1;
  for (int64_t i = 0; i < n; ++i)
    for (int32_t j = 0; j < node_out; ++j) node_feat[i * node_in + col0 + j] += out[i * node_out + j];
  return 0;
}

// Normalize of Algorithm 1 (applied to the increments, node features and
// edge features before the encoders), read as an online standardisation per
// feature column: running sums over every row seen so far,
//   stats = [n, sum_i x_ic (c < cols), sum_i x_ic^2 (c < cols)],
// with mean_c = s1_c / n and std_c = max(sqrt(max(s2_c / n - mean_c^2, 0)), eps)
// (the population deviation).  No rows seen: mean 0, std 1.
int orc_norm_accumulate(const double* x, int64_t rows, int32_t cols, double* stats) {
  if (rows < 0 || cols < 1 || !stats || (rows > 0 && !x)) return -1;
  for (int64_t i = 0; i < rows; ++i)
    for (int32_t c = 0; c < cols; ++c) {
      const double v = x[i * cols + c];
      stats[1 + c] += v;
      stats[1 + cols + c] += v * v;
    }
  stats[0] += (double)rows;
  return 0;
}

int orc_norm_apply(const double* x, int64_t rows, int32_t cols, const double* stats, double eps, double* out) {
  if (rows < 0 || cols < 1 || !stats || !(eps > 0) || (rows > 0 && (!x || !out))) return -1;
  for (int32_t c = 0; c < cols; ++c) {
    double mean = 0.0, sd = 1.0;
    if (stats[0] > 0) {
      mean = stats[1 + c] / stats[0];
      const double var = stats[1 + cols + c] / stats[0] - mean * mean;
      sd = std::sqrt(var > 0 ? var : 0.0);
      if (sd < eps) sd = eps;
    }
    for (int64_t i = 0; i < rows; ++i) out[i * cols + c] = (x[i * cols + c] - mean) / sd;
  }
  return 0;
}

}  // extern "C"

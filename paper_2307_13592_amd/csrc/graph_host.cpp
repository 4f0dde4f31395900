// Host-side graph preprocessing of libmgn: slab partition and the
// partition-local receiver / sender CSR (section "Methodology": partitions
// with a depth-1 halo; Algorithm 1 builds the send/receive masks per sample,
// here they are built once per mesh).  Counting sorts throughout: O(E + N).
#include <algorithm>
#include <cstring>
#include <vector>

#include "mgn_internal.h"

namespace mgn {

// Rank nodes by (key, id) with a stable counting sort over the key range (a
// stable comparison sort when the range is too wide), part = nparts*rank/n.
mgn_status partition_slabs(const int32_t* key, int64_t n, int32_t nparts, int32_t* part, std::string& err) {
  if (n < 0 || nparts < 1 || (n > 0 && (!key || !part))) {
    err = "mgn_partition_slabs: bad arguments";
    return MGN_E_ARG;
  }
  if (n == 0) return MGN_OK;
  int32_t kmin = key[0], kmax = key[0];
  for (int64_t i = 1; i < n; ++i) {
    kmin = std::min(kmin, key[i]);
    kmax = std::max(kmax, key[i]);
  }
  const int64_t range = (int64_t)kmax - kmin + 1;
  std::vector<int64_t> order(n);
  if (range <= 4 * n + 1024) {
    std::vector<int64_t> start(range + 1, 0);
    for (int64_t i = 0; i < n; ++i) start[key[i] - kmin + 1]++;
    for (int64_t k = 0; k < range; ++k) start[k + 1] += start[k];
    for (int64_t i = 0; i < n; ++i) order[start[key[i] - kmin]++] = i;  // ids ascending within a key
  } else {
    for (int64_t i = 0; i < n; ++i) order[i] = i;
    std::stable_sort(order.begin(), order.end(), [&](int64_t a, int64_t b) { return key[a] < key[b]; });
  }
  for (int64_t q = 0; q < n; ++q) part[order[q]] = (int32_t)(((int64_t)nparts * q) / n);
  return MGN_OK;
}

namespace {
struct Sizes {
  int64_t owned = 0, halo = 0, edges = 0;
};

mgn_status check_edges(const int32_t* send, const int32_t* recv, int64_t n_edges, const int32_t* part,
                       int64_t n_nodes, std::string& err) {
  if (n_edges < 0 || n_nodes < 0 || (n_edges > 0 && (!send || !recv)) || (n_nodes > 0 && !part)) {
    err = "graph: bad arguments";
    return MGN_E_ARG;
  }
  if (n_nodes > INT32_MAX || n_edges > INT32_MAX) {
    err = "graph: more than 2^31-1 nodes or edges";
    return MGN_E_UNSUPPORTED;
  }
  for (int64_t e = 0; e < n_edges; ++e)
    if ((uint32_t)send[e] >= (uint64_t)n_nodes || (uint32_t)recv[e] >= (uint64_t)n_nodes) {
      err = "graph: edge endpoint out of range";
      return MGN_E_GRAPH;
    }
  return MGN_OK;
}
}  // namespace

mgn_status graph_sizes(const int32_t* send, const int32_t* recv, int64_t n_edges, const int32_t* part,
                       int64_t n_nodes, int32_t p, int64_t* sizes, std::string& err) {
  mgn_status s = check_edges(send, recv, n_edges, part, n_nodes, err);
  if (s) return s;
  if (!sizes) {
    err = "mgn_graph_sizes: sizes is NULL";
    return MGN_E_ARG;
  }
  std::vector<uint8_t> mark(n_nodes, 0);  // 1 owned, 2 halo
  Sizes z;
  for (int64_t g = 0; g < n_nodes; ++g)
    if (part[g] == p) mark[g] = 1, z.owned++;
  for (int64_t e = 0; e < n_edges; ++e) {
    if (mark[recv[e]] != 1) continue;
    z.edges++;
    if (mark[send[e]] == 0) mark[send[e]] = 2, z.halo++;
  }
  sizes[0] = z.owned;
  sizes[1] = z.halo;
  sizes[2] = z.edges;
  return MGN_OK;
}

mgn_status graph_build(const int32_t* send, const int32_t* recv, int64_t n_edges, const int32_t* part,
                       int64_t n_nodes, int32_t p, int32_t* row_ptr, int32_t* send_local, int32_t* eperm,
                       int32_t* trow_ptr, int32_t* tedge, int32_t* l2g, std::string& err) {
  int64_t sz[3];
  mgn_status s = graph_sizes(send, recv, n_edges, part, n_nodes, p, sz, err);
  if (s) return s;
  const int64_t no = sz[0], nh = sz[1], ne = sz[2], nl = no + nh;
  if (!row_ptr || (ne > 0 && (!send_local || !eperm || !tedge)) || !trow_ptr || (nl > 0 && !l2g)) {
    err = "mgn_graph_build: output array is NULL";
    return MGN_E_ARG;
  }
  // global -> local: owned ids in ascending global order, then halo ids
  std::vector<int32_t> g2l(n_nodes, -1);
  int32_t next = 0;
  for (int64_t g = 0; g < n_nodes; ++g)
    if (part[g] == p) g2l[g] = next++;
  std::vector<uint8_t> halo(n_nodes, 0);
  for (int64_t e = 0; e < n_edges; ++e)
    if (part[recv[e]] == p && part[send[e]] != p) halo[send[e]] = 1;
  for (int64_t g = 0; g < n_nodes; ++g)
    if (halo[g]) g2l[g] = next++;
  for (int64_t g = 0; g < n_nodes; ++g)
    if (g2l[g] >= 0) l2g[g2l[g]] = (int32_t)g;
  // local edges in global order, then two stable counting sorts: by local
  // sender, then by local receiver -> order (receiver, sender, global id)
  std::vector<int32_t> ids;
  ids.reserve(ne);
  for (int64_t e = 0; e < n_edges; ++e)
    if (part[recv[e]] == p) ids.push_back((int32_t)e);
  std::vector<int32_t> tmp(ne);
  {
    std::vector<int64_t> cnt(nl + 1, 0);
    for (int32_t e : ids) cnt[g2l[send[e]] + 1]++;
    for (int64_t i = 0; i < nl; ++i) cnt[i + 1] += cnt[i];
    for (int32_t e : ids) tmp[cnt[g2l[send[e]]]++] = e;
  }
  {
    std::vector<int64_t> cnt(no + 1, 0);
    for (int32_t e : tmp) cnt[g2l[recv[e]] + 1]++;
    for (int64_t i = 0; i <= no; ++i) row_ptr[i] = (int32_t)cnt[i];
    for (int64_t i = 0; i < no; ++i) row_ptr[i + 1] += row_ptr[i];
    std::vector<int64_t> fill(row_ptr, row_ptr + no);
    for (int32_t e : tmp) eperm[fill[g2l[recv[e]]]++] = e;
  }
  for (int64_t i = 0; i < ne; ++i) send_local[i] = g2l[send[eperm[i]]];
  // transposed CSR: local edges grouped by sender; scanning i upwards keeps
  // each group ascending
  std::fill(trow_ptr, trow_ptr + nl + 1, 0);
  for (int64_t i = 0; i < ne; ++i) trow_ptr[send_local[i] + 1]++;
  for (int64_t n = 0; n < nl; ++n) trow_ptr[n + 1] += trow_ptr[n];
  std::vector<int32_t> pos(trow_ptr, trow_ptr + nl);
  for (int64_t i = 0; i < ne; ++i) tedge[pos[send_local[i]]++] = (int32_t)i;
  return MGN_OK;
}

// The exchange lists between parts p and q (Algorithm 1's create_masks for
// one neighbour): the halo nodes of p owned by q, by ascending halo index j
// (p's local id n_owned_p + j), with the local id each has in q (q's owned
// nodes are its l2g prefix, ascending global ids: a binary search).
mgn_status halo_masks(const int32_t* l2g_p, int64_t n_owned_p, int64_t n_halo_p, const int32_t* part,
                      int64_t n_nodes, const int32_t* l2g_q, int64_t n_owned_q, int32_t q, int32_t* recv_idx,
                      int32_t* send_rows, int64_t* count, std::string& err) {
  if (n_owned_p < 0 || n_halo_p < 0 || n_owned_q < 0 || n_nodes < 0 || !count ||
      (n_owned_p + n_halo_p > 0 && !l2g_p) || (n_owned_q > 0 && !l2g_q) || (n_nodes > 0 && !part) ||
      (n_halo_p > 0 && (!recv_idx || !send_rows))) {
    err = "mgn_halo_masks: bad arguments";
    return MGN_E_ARG;
  }
  for (int64_t i = 0; i < n_owned_q; ++i)
    if ((uint32_t)l2g_q[i] >= (uint64_t)n_nodes || (i > 0 && l2g_q[i - 1] >= l2g_q[i]) || part[l2g_q[i]] != q) {
      err = "mgn_halo_masks: q's owned nodes are not ascending global ids of part q";
      return MGN_E_GRAPH;
    }
  int64_t c = 0;
  for (int64_t j = 0; j < n_halo_p; ++j) {
    const int32_t gid = l2g_p[n_owned_p + j];
    if ((uint32_t)gid >= (uint64_t)n_nodes) {
      err = "mgn_halo_masks: halo node id out of range";
      return MGN_E_GRAPH;
    }
    if (part[gid] != q) continue;
    const int32_t* it = std::lower_bound(l2g_q, l2g_q + n_owned_q, gid);
    if (it == l2g_q + n_owned_q || *it != gid) {
      err = "mgn_halo_masks: a halo node of part q is not among q's owned nodes";
      return MGN_E_GRAPH;
    }
    recv_idx[c] = (int32_t)j;
    send_rows[c] = (int32_t)(it - l2g_q);
    ++c;
  }
  *count = c;
  return MGN_OK;
}

// Structural checks of a local graph held in host copies of the device arrays.
mgn_status graph_check(int64_t no, int64_t nh, int64_t ne, const int32_t* row_ptr, const int32_t* send,
                       const int32_t* trow, const int32_t* tedge, std::string& err) {
  const int64_t nl = no + nh;
  if (row_ptr[0] != 0 || row_ptr[no] != ne) {
    err = "graph: row_ptr must start at 0 and end at n_edges";
    return MGN_E_GRAPH;
  }
  for (int64_t r = 0; r < no; ++r)
    if (row_ptr[r + 1] < row_ptr[r]) {
      err = "graph: row_ptr is not non-decreasing";
      return MGN_E_GRAPH;
    }
  for (int64_t e = 0; e < ne; ++e)
    if (send[e] < 0 || send[e] >= nl) {
      err = "graph: sender id out of range";
      return MGN_E_GRAPH;
    }
  if (trow[0] != 0 || trow[nl] != ne) {
    err = "graph: trow_ptr must start at 0 and end at n_edges";
    return MGN_E_GRAPH;
  }
  for (int64_t n = 0; n < nl; ++n) {
    if (trow[n + 1] < trow[n]) {
      err = "graph: trow_ptr is not non-decreasing";
      return MGN_E_GRAPH;
    }
    for (int64_t i = trow[n]; i < trow[n + 1]; ++i) {
      const int32_t e = tedge[i];
      if (e < 0 || e >= ne || send[e] != n || (i > trow[n] && tedge[i - 1] >= e)) {
        err = "graph: tedge is not the ascending list of each sender's edges";
        return MGN_E_GRAPH;
      }
    }
  }
  return MGN_OK;
}

}  // namespace mgn

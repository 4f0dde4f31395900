"""Receptive-field ("cone") extraction for sampled parity at full size.

An owned node's output after K blocks depends only on nodes within K
in-edge hops and on the edges into nodes within K-1 hops (halo nodes are
leaves: their latents are inputs).  The cone of a set of centre nodes is
therefore a small partition-local graph on which the oracle reproduces those
centres' outputs exactly -- and, with the loss gradient non-zero only at the
centres, every parameter and halo gradient of the full graph.
"""
from __future__ import annotations

import numpy as np


def cone(g: dict, centers, K: int) -> dict:
    no, nh = g["n_owned"], g["n_halo"]
    row_ptr = np.asarray(g["row_ptr"], np.int64)
    send = np.asarray(g["send"], np.int64)
    dist = np.full(no + nh, K + 1, np.int64)
    centers = np.asarray(centers, np.int64)
    dist[centers] = 0
    frontier = centers
    for d in range(1, K + 1):
        fr = frontier[frontier < no]
        if fr.size == 0:
            break
        cnt = row_ptr[fr + 1] - row_ptr[fr]
        idx = np.repeat(row_ptr[fr], cnt) + (np.arange(cnt.sum()) - np.repeat(np.cumsum(cnt) - cnt, cnt))
        nb = np.unique(send[idx])
        nb = nb[dist[nb] > d]
        dist[nb] = d
        frontier = nb
    nodes = np.nonzero(dist <= K)[0]
    owned = nodes[nodes < no]
    halo = nodes[nodes >= no]
    sub_id = np.full(no + nh, -1, np.int64)
    sub_id[owned] = np.arange(owned.size)
    sub_id[halo] = owned.size + np.arange(halo.size)
    # receivers within K-1 hops keep all their in-edges
    full_rx = owned[dist[owned] <= K - 1]
    cnt_all = np.zeros(owned.size, np.int64)
    cnt_all[sub_id[full_rx]] = row_ptr[full_rx + 1] - row_ptr[full_rx]
    rp = np.concatenate([[0], np.cumsum(cnt_all)])
    # local edge ids of the kept edges, in the sub-graph's receiver order
    starts = row_ptr[owned]
    idx = np.repeat(starts, cnt_all) + (np.arange(rp[-1]) - np.repeat(rp[:-1], cnt_all))
    s_sub = sub_id[send[idx]]
    # within a receiver, order by sub-graph sender id (kept monotone: owned and
    # halo ids keep their relative order in the sub-graph)
    assert np.all(s_sub >= 0)
    return dict(n_owned=int(owned.size), n_halo=int(halo.size), n_edges=int(idx.size),
                row_ptr=rp.astype(np.int32), send=s_sub.astype(np.int32),
                owned=owned, halo=halo - no, edges=idx, centers_sub=sub_id[centers])


def cone_digest(c: dict, sub: dict, params) -> str:
    """sha256 over a cone's graph and its inputs (node and edge features, halo
    latents, loss gradient, parameters), in that order: ties a stored result
    to the inputs that regenerate it."""
    import hashlib
    h = hashlib.sha256()
    for a in (c["row_ptr"], c["send"], sub["nf"], sub["ef"], sub["halo"], sub["d_out"], params):
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


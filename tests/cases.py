"""Small helpers shared by the tests: local graphs and inputs of tiny meshes."""
from __future__ import annotations

import numpy as np

import synth
import oracle


def brute_graph(send, recv, part, n_nodes, p):
    """Partition-local graph written out from its definition with Python sets
    and sorts (owned receiver edges; halo = their non-owned senders)."""
    send = np.asarray(send, np.int64)
    recv = np.asarray(recv, np.int64)
    part = np.asarray(part)
    owned = [g for g in range(n_nodes) if part[g] == p]
    local_edges = [e for e in range(len(send)) if part[recv[e]] == p]
    halo = sorted({int(send[e]) for e in local_edges if part[send[e]] != p})
    l2g = owned + halo
    g2l = {g: i for i, g in enumerate(l2g)}
    order = sorted(local_edges, key=lambda e: (g2l[int(recv[e])], g2l[int(send[e])], e))
    row_ptr = [0] * (len(owned) + 1)
    for e in order:
        row_ptr[g2l[int(recv[e])] + 1] += 1
    row_ptr = np.cumsum(row_ptr)
    send_local = [g2l[int(send[e])] for e in order]
    tedge = []
    trow = [0]
    for n in range(len(l2g)):
        mine = [i for i, s in enumerate(send_local) if s == n]
        tedge += mine
        trow.append(len(tedge))
    return dict(n_owned=len(owned), n_halo=len(halo), n_edges=len(order),
                row_ptr=np.asarray(row_ptr, np.int32), send=np.asarray(send_local, np.int32),
                eperm=np.asarray(order, np.int32), trow_ptr=np.asarray(trow, np.int32),
                tedge=np.asarray(tedge, np.int32), l2g=np.asarray(l2g, np.int32))


def local_case(mesh, p, latent, K, depth, seed, part=None, halo_scale=1.0):
    """Oracle-built local graph of partition p plus its float64 inputs."""
    if part is None:
        part = oracle.partition(mesh.key, mesh.nparts) if mesh.part is None else mesh.part
    g = oracle.graph_build(mesh.send, mesh.recv, part, mesh.n_nodes, p)
    shapes = synth.param_shapes(latent, K, depth)
    params = synth.init_params(shapes, seed).astype(np.float64)
    nf = synth.node_features(mesh, seed)[g["l2g"][:g["n_owned"]]].astype(np.float64)
    ef = synth.edge_features(mesh)[g["eperm"]].astype(np.float64)
    halo = synth.halo_latents(K, g["n_halo"], latent, seed).astype(np.float64) * halo_scale
    rng = np.random.default_rng([seed, 99])
    d_out = rng.standard_normal((g["n_owned"], 5))
    cfg = oracle.ModelCfg(latent, K, depth)
    return dict(g=g, cfg=cfg, shapes=shapes, params=params, nf=nf, ef=ef, halo=halo, d_out=d_out, part=part)

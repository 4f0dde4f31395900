"""The input generator: sizes against closed forms, determinism, region
consistency.  (The generator draws inputs only; nothing here is the method.)"""
import numpy as np

import synth
from synth import meshes


def _undirected_ok(m):
    a = m.send.astype(np.int64) * m.n_nodes + m.recv
    b = m.recv.astype(np.int64) * m.n_nodes + m.send
    assert np.array_equal(np.sort(a), np.sort(b)), "every directed edge needs its reverse"
    assert len(np.unique(a)) == len(a), "no duplicate directed edges"
    assert not np.any(m.send == m.recv)


def test_hex_counts():
    m = meshes.hex_lattice(16)
    assert m.n_nodes == 4096
    assert m.n_edges == 2 * 3 * 16 * 16 * 15 == 23040
    _undirected_ok(m)
    deg = np.bincount(m.recv, minlength=m.n_nodes)
    assert deg.max() == 6 and deg.min() == 3


def test_sector_counts_and_degree():
    m = meshes.sector(6, 16, 10, 4, seed=7)
    assert m.n_nodes == 6 * 16 * 10
    assert m.n_edges == meshes.edge_count_sector(6, 16, 10)
    _undirected_ok(m)
    deg = np.bincount(m.recv, minlength=m.n_nodes)
    assert deg.max() == 14          # interior nodes of the Kuhn split


def test_region_matches_full_mesh():
    full = meshes.sector(5, 16, 7, 4, seed=3)
    reg = meshes.sector(5, 16, 7, 4, seed=3, t_lo=3, t_hi=8)
    off = 3 * 5 * 7
    sl = slice(off, off + reg.n_nodes)
    assert np.array_equal(full.coords[sl], reg.coords)
    assert np.array_equal(full.node_type[sl], reg.node_type)
    assert np.array_equal(synth.node_features(full, 3)[sl], synth.node_features(reg, 3))
    assert np.array_equal(synth.targets(full, 3)[sl], synth.targets(reg, 3))
    # region edges = full-mesh edges with both ends inside, same relative order
    inside = (full.send >= off) & (full.send < off + reg.n_nodes) & (full.recv >= off) & (full.recv < off + reg.n_nodes)
    fe = set(zip((full.send[inside] - off).tolist(), (full.recv[inside] - off).tolist()))
    re = set(zip(reg.send.tolist(), reg.recv.tolist()))
    assert fe == re


def test_determinism():
    a = synth.make_case(synth.CONFIGS["C1"])
    b = synth.make_case(synth.CONFIGS["C1"])
    for k in ("node_feat", "edge_feat", "target", "params"):
        assert np.array_equal(getattr(a, k), getattr(b, k))
    assert a.params.shape[0] == 72517


def test_param_counts():
    for l, K, D, n in ((64, 2, 2, 72517), (128, 15, 2, 1788549), (256, 15, 3, 9287173)):
        shapes = synth.param_shapes(l, K, D)
        assert sum(int(np.prod(s)) for _, _, s in shapes) == n


def test_features_shapes():
    m = meshes.sector(6, 16, 10, 4, seed=7)
    f = synth.node_features(m, 7)
    assert f.shape == (m.n_nodes, 11) and f.dtype == np.float32
    assert np.all(f[:, 8:].sum(1) == 1)
    e = synth.edge_features(m)
    assert e.shape == (m.n_edges, 4)
    assert np.all(e[:, 3] > 0)

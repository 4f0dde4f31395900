"""Pins of the oracle's integer work: partition and partition-local graph,
against brute force written from the definitions (section "Methodology":
METIS-style parts, depth-1 halo of directly connected nodes)."""
import numpy as np
import pytest

import oracle
import synth
from synth import meshes
from cases import brute_graph


def test_partition_brute_force():
    rng = np.random.default_rng(0)
    for n, P in ((1, 1), (7, 3), (100, 4), (1000, 8)):
        key = rng.integers(0, 5, n).astype(np.int32)
        order = sorted(range(n), key=lambda i: (key[i], i))
        want = np.empty(n, np.int32)
        for q, i in enumerate(order):
            want[i] = (P * q) // n
        assert np.array_equal(oracle.partition(key, P), want)


def test_partition_sector_is_theta_slabs():
    m = meshes.sector(5, 16, 7, 4, seed=3)
    part = oracle.partition(m.key, 4)
    assert np.array_equal(part, m.key // 4)
    reg = meshes.sector(5, 16, 7, 4, seed=3, t_lo=3, t_hi=8)
    assert np.array_equal(reg.part, part[3 * 35:9 * 35])


@pytest.mark.parametrize("mesh,P", [
    (meshes.hex_lattice(5), 1),
    (meshes.hex_lattice(6), 1),
    (meshes.sector(4, 12, 5, 4, seed=1), 4),
    (meshes.delaunay_box(6, 5, 4, seed=3), 1),
])
def test_graph_build_brute_force(mesh, P):
    part = oracle.partition(mesh.key, P)
    for p in range(P):
        g = oracle.graph_build(mesh.send, mesh.recv, part, mesh.n_nodes, p)
        b = brute_graph(mesh.send, mesh.recv, part, mesh.n_nodes, p)
        for k in b:
            if isinstance(b[k], np.ndarray):
                assert np.array_equal(g[k], b[k]), k
            else:
                assert g[k] == b[k], k


def test_graph_random_partition_brute_force():
    m = meshes.delaunay_box(6, 6, 5, seed=4)
    rng = np.random.default_rng(5)
    part = rng.integers(0, 3, m.n_nodes).astype(np.int32)
    for p in range(3):
        g = oracle.graph_build(m.send, m.recv, part, m.n_nodes, p)
        b = brute_graph(m.send, m.recv, part, m.n_nodes, p)
        for k in b:
            assert np.array_equal(np.asarray(g[k]), np.asarray(b[k])), k


def test_graph_invariants_sector_partition():
    """In-degree segments, halo = non-owned senders, every owned node once."""
    m = meshes.sector(6, 16, 10, 4, seed=7)
    part = oracle.partition(m.key, 4)
    seen = np.zeros(m.n_nodes, int)
    for p in range(4):
        g = oracle.graph_build(m.send, m.recv, part, m.n_nodes, p)
        no = g["n_owned"]
        owned = g["l2g"][:no]
        seen[owned] += 1
        indeg = np.bincount(m.recv, minlength=m.n_nodes)[owned]
        assert np.array_equal(np.diff(g["row_ptr"]), indeg)
        assert np.all(part[g["l2g"][no:]] != p)
        # an interior slab has two neighbours, each contributing one theta layer
        if p in (1, 2):
            assert g["n_halo"] == 2 * 6 * 10
        # gathering through the transposed CSR visits every local edge once
        assert np.array_equal(np.sort(g["tedge"]), np.arange(g["n_edges"]))
    assert np.all(seen == 1)


def test_c3_local_sizes():
    """The 1M-owned-node slab: sizes stated for the configuration."""
    case = synth.CONFIGS["C3"]
    m = case.build_mesh(True)
    g = oracle.graph_build(m.send, m.recv, m.part, m.n_nodes, case.part)
    assert (g["n_owned"], g["n_halo"], g["n_edges"]) == (1_000_000, 50_000, 13_824_160)


def test_edge_features_match_generator():
    m = meshes.sector(4, 12, 5, 4, seed=1)
    want = oracle.edge_features(m.coords, m.send, m.recv, m.h)
    got = synth.edge_features(m)
    np.testing.assert_allclose(got, want, rtol=2e-7, atol=1e-6)
    # sender minus receiver: reversing the edge flips the displacement
    n = m.n_edges // 2
    np.testing.assert_array_equal(got[:n, :3], -got[n:, :3])

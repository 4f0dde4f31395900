"""libmgn without a GPU: the shared library loads and exports every entry
point include/mgn.h declares; its host-side graph preprocessing agrees bit
for bit with the oracle's; parameter layout sizes agree; argument and state
errors are reported before anything is launched."""
import os
import re

import numpy as np
import pytest

import oracle
import synth
from synth import meshes
import paper_2307_13592_amd as mgn

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_exports_every_declared_symbol():
    hdr = open(os.path.join(ROOT, "include", "mgn.h")).read()
    declared = set(re.findall(r"^\S[^;(]*?\b(mgn_\w+)\s*\(", hdr, re.M))
    assert declared == set(mgn.EXPORTS)
    L = mgn.lib()
    for name in declared:
        assert getattr(L, name) is not None


@pytest.mark.parametrize("mesh,P", [
    (meshes.hex_lattice(6), 1),
    (meshes.sector(4, 12, 5, 4, seed=1), 4),
    (meshes.sector(6, 16, 10, 4, seed=7), 4),
    (meshes.delaunay_box(8, 7, 6, seed=3), 1),
])
def test_graph_build_matches_oracle(mesh, P):
    part_o = oracle.partition(mesh.key, P)
    part_m = mgn.mgn_partition_slabs(mesh.key, P)
    assert np.array_equal(part_o, part_m)
    for p in range(P):
        go = oracle.graph_build(mesh.send, mesh.recv, part_o, mesh.n_nodes, p)
        gm = mgn.mgn_graph_build(mesh.send, mesh.recv, part_m, mesh.n_nodes, p)
        for k in go:
            assert np.array_equal(np.asarray(go[k]), np.asarray(gm[k])), k


def test_graph_build_random_partition_matches_oracle():
    m = meshes.delaunay_box(9, 8, 7, seed=5)
    part = np.random.default_rng(1).integers(0, 5, m.n_nodes).astype(np.int32)
    for p in range(5):
        go = oracle.graph_build(m.send, m.recv, part, m.n_nodes, p)
        gm = mgn.mgn_graph_build(m.send, m.recv, part, m.n_nodes, p)
        for k in go:
            assert np.array_equal(np.asarray(go[k]), np.asarray(gm[k])), k


def test_partition_matches_oracle_wide_keys():
    rng = np.random.default_rng(2)
    for n, P, hi in ((1000, 7, 5), (5000, 3, 10 ** 9), (17, 4, 2)):
        key = rng.integers(-hi, hi, n).astype(np.int32)
        assert np.array_equal(oracle.partition(key, P), mgn.mgn_partition_slabs(key, P))


def test_c3_graph_build_matches_oracle():
    """The 1M-owned-node slab at full size, bit-exact."""
    cfg = synth.CONFIGS["C3"]
    m = cfg.build_mesh(True)
    go = oracle.graph_build(m.send, m.recv, m.part, m.n_nodes, cfg.part)
    gm = mgn.mgn_graph_build(m.send, m.recv, m.part, m.n_nodes, cfg.part)
    for k in go:
        assert np.array_equal(np.asarray(go[k]), np.asarray(gm[k])), k


def test_param_count_matches_oracle_and_layout():
    for l, K, D in ((64, 2, 2), (128, 15, 2), (256, 15, 3), (64, 0, 3)):
        h = mgn.mgn_create(l, K, D)
        try:
            n = mgn.mgn_param_count(h)
        finally:
            mgn.mgn_destroy(h)
        assert n == oracle.param_count(oracle.ModelCfg(l, K, D))
        assert n == sum(int(np.prod(s)) for _, _, s in synth.param_shapes(l, K, D))


def test_create_rejects_unsupported():
    for kw in (dict(latent=96), dict(depth=4), dict(node_out=17), dict(node_in=0), dict(precision=7),
               dict(n_blocks=-1)):
        args = dict(latent=64, n_blocks=2, depth=2)
        args.update(kw)
        with pytest.raises(mgn.MgnError) as e:
            mgn.mgn_create(**args)
        assert e.value.status == mgn.MGN_E_UNSUPPORTED
    with pytest.raises(mgn.MgnError) as e:
        mgn.mgn_create(64, 2, 2, ln_eps=0.0)
    assert e.value.status == mgn.MGN_E_ARG


def test_graph_errors():
    m = meshes.hex_lattice(3)
    part = np.zeros(m.n_nodes, np.int32)
    bad = m.send.copy()
    bad[5] = m.n_nodes + 3
    with pytest.raises(mgn.MgnError) as e:
        mgn.mgn_graph_sizes(bad, m.recv, part, m.n_nodes, 0)
    assert e.value.status == mgn.MGN_E_GRAPH
    with pytest.raises(mgn.MgnError) as e:
        mgn.mgn_partition_slabs(np.zeros(4, np.int32), 0)
    assert e.value.status == mgn.MGN_E_ARG


def test_state_errors_before_any_launch():
    """Forward before set_params / validation, backward before forward: the
    status comes back without touching the device."""
    import ctypes as C
    h = mgn.mgn_create(64, 1, 2)
    try:
        g = mgn.mgn_graph(4, 0, 0, C.c_void_p(256), C.c_void_p(512), C.c_void_p(768), C.c_void_p(1024))
        L = mgn.lib()
        st = L.mgn_forward(h, C.byref(g), None, None, None, None, None, 0, None)
        assert st == mgn.MGN_E_STATE and "never set" in mgn.mgn_last_error(h)
        st = L.mgn_backward(h, None, C.c_void_p(256), 0, None, None)
        assert st == mgn.MGN_E_STATE and "no forward" in mgn.mgn_last_error(h)
        n = C.c_size_t()
        assert L.mgn_workspace_size(h, C.byref(g), C.byref(n)) == mgn.MGN_OK and n.value > 0
        g.n_owned = -1
        assert L.mgn_workspace_size(h, C.byref(g), C.byref(n)) == mgn.MGN_E_ARG
        g.n_owned = 4
        g.row_ptr = C.c_void_p(258)     # misaligned
        assert L.mgn_workspace_size(h, C.byref(g), C.byref(n)) == mgn.MGN_E_ARG
    finally:
        mgn.mgn_destroy(h)
    assert mgn.lib().mgn_mse_grad(None, None, None, 3, 0, None, None, None) == mgn.MGN_E_ARG


def test_recompute_setting():
    """Edge-stream checkpointing is a bf16-mode setting; it shrinks the
    workspace of a graph with several blocks."""
    import ctypes as C
    L = mgn.lib()
    h32 = mgn.mgn_create(64, 4, 2)
    try:
        assert L.mgn_set_recompute(h32, 2, 0) == mgn.MGN_E_UNSUPPORTED
        assert L.mgn_set_recompute(h32, 0, 0) == mgn.MGN_OK
    finally:
        mgn.mgn_destroy(h32)
    h = mgn.mgn_create(64, 8, 2, mgn.MGN_BF16)
    try:
        assert L.mgn_set_recompute(h, -1, 0) == mgn.MGN_E_ARG
        assert L.mgn_set_recompute(h, 1, -5) == mgn.MGN_E_ARG
        g = mgn.mgn_graph(1000, 0, 20000, C.c_void_p(256), C.c_void_p(512), C.c_void_p(768), C.c_void_p(1024))
        n0, n4 = C.c_size_t(), C.c_size_t()
        assert L.mgn_workspace_size(h, C.byref(g), C.byref(n0)) == mgn.MGN_OK
        assert L.mgn_set_recompute(h, 4, 0) == mgn.MGN_OK
        assert L.mgn_workspace_size(h, C.byref(g), C.byref(n4)) == mgn.MGN_OK
        # 8 edge-latent copies down to 2 checkpoints + 1 working copy (bf16, 64 wide)
        assert n0.value - n4.value >= 5 * 20000 * 64 * 2
    finally:
        mgn.mgn_destroy(h)


def test_norm_argument_checks():
    """Normalize's entry points reject bad sizes, eps and pointers on the host
    (no device work is issued)."""
    L = mgn.lib()
    st, wk, x = C_vp(4096), C_vp(8192), C_vp(12288)
    assert L.mgn_norm_accumulate(x, -1, 4, st, wk, None) == mgn.MGN_E_ARG
    assert L.mgn_norm_accumulate(x, 10, 0, st, wk, None) == mgn.MGN_E_ARG
    assert L.mgn_norm_accumulate(x, 10, mgn.MGN_NORM_MAX_COLS + 1, st, wk, None) == mgn.MGN_E_ARG
    assert L.mgn_norm_accumulate(x, 10, 4, None, wk, None) == mgn.MGN_E_ARG
    assert L.mgn_norm_accumulate(x, 10, 4, st, None, None) == mgn.MGN_E_ARG
    assert L.mgn_norm_accumulate(None, 10, 4, st, wk, None) == mgn.MGN_E_ARG
    assert L.mgn_norm_accumulate(x, 10, 4, C_vp(4100), wk, None) == mgn.MGN_E_ARG  # stats not 8-byte aligned
    assert L.mgn_norm_accumulate(None, 0, 4, st, wk, None) == mgn.MGN_OK  # no rows: nothing to do
    assert L.mgn_norm_apply(x, 10, 4, st, 0.0, x, None) == mgn.MGN_E_ARG
    assert L.mgn_norm_apply(x, 10, 4, st, -1.0, x, None) == mgn.MGN_E_ARG
    assert L.mgn_norm_apply(x, 10, 65, st, 1e-8, x, None) == mgn.MGN_E_ARG
    assert L.mgn_norm_apply(x, 10, 4, st, 1e-8, None, None) == mgn.MGN_E_ARG
    assert L.mgn_norm_apply(x, 10, 4, None, 1e-8, x, None) == mgn.MGN_E_ARG
    assert L.mgn_norm_apply(None, 0, 4, st, 1e-8, None, None) == mgn.MGN_OK


def C_vp(v):
    import ctypes as C
    return C.c_void_p(v)


def test_h1_stash_setting():
    """The first-Linear stash adds one bf16 E x l slot per kept block to the
    row-split plan (at most K), and the kept blocks share one node-projection
    slot (fp32, 2l per node) instead of one each; nothing changes for the
    streaming plans (which keep every block's anyway) or with checkpointing."""
    import ctypes as C
    L = mgn.lib()
    g = mgn.mgn_graph(1000, 0, 20000, C.c_void_p(256), C.c_void_p(512), C.c_void_p(768), C.c_void_p(1024))

    def ws(h):
        n = C.c_size_t()
        assert L.mgn_workspace_size(h, C.byref(g), C.byref(n)) == mgn.MGN_OK
        return n.value

    h = mgn.mgn_create(64, 6, 2, mgn.MGN_BF16)
    try:
        assert L.mgn_set_h1_stash(h, -1) == mgn.MGN_E_ARG
        n0 = ws(h)
        assert L.mgn_set_h1_stash(h, 2) == mgn.MGN_OK
        n2 = ws(h)
        assert L.mgn_set_h1_stash(h, 50) == mgn.MGN_OK
        n6 = ws(h)
        slot, proj = 20000 * 64 * 2, 1000 * 2 * 64 * 4
        d2, d6 = 2 * slot - proj, 6 * slot - 5 * proj
        assert d2 <= n2 - n0 <= d2 + 1024 and d6 <= n6 - n0 <= d6 + 1024
        assert L.mgn_set_recompute(h, 2, 0) == mgn.MGN_OK
        n_lean = ws(h)
        assert L.mgn_set_h1_stash(h, 0) == mgn.MGN_OK
        assert ws(h) == n_lean
    finally:
        mgn.mgn_destroy(h)
    h = mgn.mgn_create(256, 3, 3, mgn.MGN_BF16)  # streaming kernels
    try:
        n0 = ws(h)
        assert L.mgn_set_h1_stash(h, 3) == mgn.MGN_OK
        assert ws(h) == n0
    finally:
        mgn.mgn_destroy(h)
    assert L.mgn_set_h1_stash(None, 1) == mgn.MGN_E_ARG


@pytest.mark.parametrize("mesh,P,random", [
    (meshes.sector(6, 16, 10, 4, seed=7), 4, False),
    (meshes.delaunay_box(9, 8, 7, seed=5), 5, True),
])
def test_halo_masks_brute_force(mesh, P, random):
    """Exchange lists of every (part, owner) pair against their definition
    (halo nodes of p owned by q, ascending halo index; q's local id of each),
    written with Python dicts; every halo node is in exactly one owner's list."""
    if random:
        part = np.random.default_rng(3).integers(0, P, mesh.n_nodes).astype(np.int32)
    else:
        part = mgn.mgn_partition_slabs(mesh.key, P)
    gs = [mgn.mgn_graph_build(mesh.send, mesh.recv, part, mesh.n_nodes, p) for p in range(P)]
    for p in range(P):
        no_p = gs[p]["n_owned"]
        halo_g = [int(x) for x in gs[p]["l2g"][no_p:]]
        covered = 0
        for q in range(P):
            if q == p:
                continue
            recv, send = mgn.mgn_halo_masks(gs[p]["l2g"], no_p, part, gs[q]["l2g"], gs[q]["n_owned"], q)
            pos = {int(gid): i for i, gid in enumerate(gs[q]["l2g"][:gs[q]["n_owned"]])}
            want_recv = [j for j, gid in enumerate(halo_g) if part[gid] == q]
            want_send = [pos[halo_g[j]] for j in want_recv]
            assert recv.tolist() == want_recv and send.tolist() == want_send
            covered += len(want_recv)
        assert covered == len(halo_g)


def test_halo_masks_errors():
    mesh = meshes.sector(4, 12, 5, 4, seed=1)
    part = mgn.mgn_partition_slabs(mesh.key, 4)
    g0 = mgn.mgn_graph_build(mesh.send, mesh.recv, part, mesh.n_nodes, 0)
    g1 = mgn.mgn_graph_build(mesh.send, mesh.recv, part, mesh.n_nodes, 1)
    bad = g1["l2g"].copy()
    bad[[0, 1]] = bad[[1, 0]]  # q's owned list no longer ascending
    with pytest.raises(mgn.MgnError) as e:
        mgn.mgn_halo_masks(g0["l2g"], g0["n_owned"], part, bad, g1["n_owned"], 1)
    assert e.value.status == mgn.MGN_E_GRAPH
    with pytest.raises(mgn.MgnError) as e:  # q = 2 does not own g1's nodes
        mgn.mgn_halo_masks(g0["l2g"], g0["n_owned"], part, g1["l2g"], g1["n_owned"], 2)
    assert e.value.status == mgn.MGN_E_GRAPH


def test_staged_state_errors_before_any_launch():
    """The stages of a staged step called out of order, and the exchanges
    without a step in progress: MGN_E_STATE, nothing launched."""
    import ctypes as C
    L = mgn.lib()
    h = mgn.mgn_create(64, 2, 2)
    try:
        fake = C.c_void_p(4096)
        for call, what in ((lambda: L.mgn_forward_block(h, None), "no forward block"),
                           (lambda: L.mgn_forward_end(h, None), "not all run"),
                           (lambda: L.mgn_backward_begin(h, fake, fake, 0, None, None), "no forward"),
                           (lambda: L.mgn_backward_block(h, None), "no backward block"),
                           (lambda: L.mgn_backward_end(h, None), "not all run"),
                           (lambda: L.mgn_copy_latents(h, fake, fake, 3, fake, 5, None), "no forward"),
                           (lambda: L.mgn_add_latent_grads(h, fake, 5, fake, fake, 3, None), "no backward")):
            assert call() == mgn.MGN_E_STATE
            assert what in mgn.mgn_last_error(h)
        assert L.mgn_copy_latents(h, fake, fake, -1, fake, 5, None) == mgn.MGN_E_ARG
        assert L.mgn_copy_latents(h, None, fake, 3, fake, 5, None) == mgn.MGN_E_ARG
        assert L.mgn_copy_latents(h, fake, fake, 0, None, 0, None) == mgn.MGN_OK  # nothing to copy
        assert L.mgn_forward_block(None, None) == mgn.MGN_E_ARG
    finally:
        mgn.mgn_destroy(h)


def test_lockstep_argument_errors():
    """mgn_lockstep_forward / _backward reject bad part counts and links
    before anything is launched."""
    import ctypes as C
    L = mgn.lib()
    h0, h1 = mgn.mgn_create(64, 2, 2), mgn.mgn_create(64, 2, 2)
    h3 = mgn.mgn_create(128, 2, 2)
    try:
        ms = (C.c_void_p * 2)(h0.value, h1.value)
        fake = C.c_void_p(4096)
        bad = (mgn.mgn_halo_link * 1)(mgn.mgn_halo_link(0, 5, fake, fake, 3))       # owner out of range
        assert L.mgn_lockstep_backward(2, ms, None, None, 0, None, bad, 1, None) == mgn.MGN_E_ARG
        self_link = (mgn.mgn_halo_link * 1)(mgn.mgn_halo_link(1, 1, fake, fake, 3))
        assert L.mgn_lockstep_backward(2, ms, None, None, 0, None, self_link, 1, None) == mgn.MGN_E_ARG
        assert L.mgn_lockstep_backward(0, ms, None, None, 0, None, None, 0, None) == mgn.MGN_E_ARG
        mixed = (C.c_void_p * 2)(h0.value, h3.value)                                  # latent 64 vs 128
        ok = (mgn.mgn_halo_link * 1)(mgn.mgn_halo_link(0, 1, fake, fake, 3))
        assert L.mgn_lockstep_backward(2, mixed, None, None, 0, None, ok, 1, None) == mgn.MGN_E_ARG
        assert "latent" in mgn.mgn_last_error(None)
        # no forward before the backward: each part reports it
        d = (C.c_void_p * 2)(fake.value, fake.value)
        assert L.mgn_lockstep_backward(2, ms, d, fake, 0, d, ok, 1, None) == mgn.MGN_E_STATE
    finally:
        for h in (h0, h1, h3):
            mgn.mgn_destroy(h)

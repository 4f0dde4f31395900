"""Pins of the oracle's network arithmetic against things other than itself:
an independent library-layer formulation with autograd, finite differences,
node-permutation equivariance, partition consistency with exact halos,
exact linearity of the backward pass, a dense incidence-matrix product for the
receiver sum, and LayerNorm's closed-form row mean."""
import numpy as np
import pytest
import torch

import oracle
import synth
from synth import meshes
import torch_ref
from cases import local_case


def _rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    den = np.abs(b).max() if b.size else 0.0
    return float(np.abs(a - b).max() / den) if den > 0 else float(np.abs(a - b).max() if a.size else 0.0)


def _segments(shapes):
    off = 0
    for name, _, shape in shapes:
        n = int(np.prod(shape))
        yield name, slice(off, off + n)
        off += n


CASES = [
    ("hex4", lambda: meshes.hex_lattice(4), 0, 8, 2, 2),
    ("hex5_D3", lambda: meshes.hex_lattice(5), 0, 8, 2, 3),
    ("sector_p1_K3", lambda: meshes.sector(3, 8, 4, 4, seed=2), 1, 8, 3, 3),
    ("sector_p0_K2", lambda: meshes.sector(3, 8, 4, 4, seed=2), 0, 16, 2, 2),
    ("delaunay", lambda: meshes.delaunay_box(5, 4, 4, seed=6), 0, 16, 1, 2),
]


@pytest.mark.parametrize("name,mk,p,l,K,D", CASES, ids=[c[0] for c in CASES])
def test_matches_torch_layers(name, mk, p, l, K, D):
    c = local_case(mk(), p, l, K, D, seed=3)
    g = c["g"]
    r = oracle.step(c["cfg"], g, c["params"], c["nf"], c["ef"], c["halo"], c["d_out"])
    out, dp, dh = torch_ref.run(l, K, D, c["shapes"], g, c["params"], c["nf"], c["ef"], c["halo"], c["d_out"])
    assert _rel(r["out"], out) < 1e-12
    for nm, sl in _segments(c["shapes"]):
        assert _rel(r["d_params"][sl], dp[sl]) < 1e-11, nm
    if g["n_halo"]:
        assert _rel(r["d_halo"], dh) < 1e-11
        assert np.abs(dh).max() > 0


@pytest.mark.parametrize("name,mk,p,l,K,D", CASES[:3], ids=[c[0] for c in CASES[:3]])
def test_bf16_mode_matches_torch_bfloat16(name, mk, p, l, K, D):
    """The oracle's mixed-precision mode against torch's own bfloat16
    rounding at the same points (independent formulation)."""
    c = local_case(mk(), p, l, K, D, seed=3)
    cfg = oracle.ModelCfg(l, K, D, bf16=True)
    r = oracle.step(cfg, c["g"], c["params"], c["nf"], c["ef"], c["halo"], c["d_out"])
    out, dp, dh = torch_ref.run(l, K, D, c["shapes"], c["g"], c["params"], c["nf"], c["ef"], c["halo"],
                                c["d_out"], bf16=True)
    assert _rel(r["out"], out) < 1e-12
    for nm, sl in _segments(c["shapes"]):
        assert _rel(r["d_params"][sl], dp[sl]) < 1e-10, nm
    if c["g"]["n_halo"]:
        assert _rel(r["d_halo"], dh) < 1e-10
    # and it is a different function from the float64 one
    r64 = oracle.step(c["cfg"], c["g"], c["params"], c["nf"], c["ef"], c["halo"], c["d_out"])
    assert _rel(r["out"], r64["out"]) > 1e-5


def test_edgeless_K0_is_encoder_then_decoder():
    """K = 0 and no edges: the network is nn.Sequential(encoder, decoder)."""
    l, D = 16, 3
    shapes = synth.param_shapes(l, 0, D)
    params = synth.init_params(shapes, 5).astype(np.float64)
    rng = np.random.default_rng(1)
    n = 37
    nf = rng.standard_normal((n, 11))
    g = dict(n_owned=n, n_halo=0, n_edges=0, row_ptr=np.zeros(n + 1, np.int32), send=np.zeros(0, np.int32))
    d_out = rng.standard_normal((n, 5))
    r = oracle.step(oracle.ModelCfg(l, 0, D), g, params, nf, np.zeros((0, 4)), None, d_out)
    model = torch_ref.TorchMGN(l, 0, D)
    model.load_flat(params, shapes)
    seq = torch.nn.Sequential(model.enc_node, model.dec)
    out = seq(torch.as_tensor(nf))
    out.backward(torch.as_tensor(d_out))
    assert _rel(r["out"], out.detach().numpy()) < 1e-13
    dp = model.flat_grad().numpy()
    assert _rel(r["d_params"], dp) < 1e-12
    ee = [sl for nm, sl in _segments(shapes) if nm.startswith("enc_edge")]
    assert all(np.all(r["d_params"][sl] == 0) for sl in ee)


@pytest.mark.parametrize("D", [2, 3])
def test_finite_differences(D):
    """Central differences, h = 1e-6, over every parameter and halo entry of a
    partitioned tiny sector (l = 8, K = 2)."""
    c = local_case(meshes.sector(3, 8, 3, 4, seed=4), 1, 8, 2, D, seed=11)
    g, cfg = c["g"], c["cfg"]
    assert g["n_halo"] > 0
    d_out = c["d_out"]
    r = oracle.step(cfg, g, c["params"], c["nf"], c["ef"], c["halo"], d_out)

    def L(params, halo):
        o = oracle.step(cfg, g, params, c["nf"], c["ef"], halo)["out"]
        return float((o * d_out).sum())

    h = 1e-6
    P = c["params"]
    fd = np.empty_like(P)
    for i in range(P.size):
        a, b = P.copy(), P.copy()
        a[i] += h
        b[i] -= h
        fd[i] = (L(a, c["halo"]) - L(b, c["halo"])) / (2 * h)
    for nm, sl in _segments(c["shapes"]):
        assert _rel(fd[sl], r["d_params"][sl]) < 1e-6, nm
    H = c["halo"]
    fdh = np.empty_like(H)
    it = np.nditer(H, flags=["multi_index"])
    for _ in it:
        a, b = H.copy(), H.copy()
        a[it.multi_index] += h
        b[it.multi_index] -= h
        fdh[it.multi_index] = (L(P, a) - L(P, b)) / (2 * h)
    assert _rel(fdh, r["d_halo"]) < 1e-6


def test_permutation_equivariance():
    m = meshes.delaunay_box(5, 5, 4, seed=9)
    c = local_case(m, 0, 16, 2, 2, seed=4)
    r = oracle.step(c["cfg"], c["g"], c["params"], c["nf"], c["ef"], None, c["d_out"])
    rng = np.random.default_rng(2)
    pi = rng.permutation(m.n_nodes).astype(np.int32)        # new id of old node i
    inv = np.argsort(pi)
    part = np.zeros(m.n_nodes, np.int32)
    g2 = oracle.graph_build(pi[m.send], pi[m.recv], part, m.n_nodes, 0)
    # local ids of the relabelled graph are the new ids; inputs follow
    nf_full = synth.node_features(m, 4).astype(np.float64)
    ef_full = synth.edge_features(m).astype(np.float64)
    nf2 = nf_full[inv]
    ef2 = ef_full[g2["eperm"]]
    d_out_full = np.empty_like(c["d_out"])
    d_out_full[c["g"]["l2g"]] = c["d_out"]
    r2 = oracle.step(c["cfg"], g2, c["params"], nf2, ef2, None, d_out_full[inv])
    out_full = np.empty_like(r["out"])
    out_full[c["g"]["l2g"]] = r["out"]
    assert _rel(r2["out"], out_full[inv]) < 1e-12
    assert _rel(r2["d_params"], r["d_params"]) < 1e-11


def test_partition_consistency():
    """Each partition fed the unpartitioned network's halo latents reproduces
    the unpartitioned outputs and edge latents of everything it owns."""
    m = meshes.sector(6, 16, 10, 4, seed=7)
    K, l, D = 3, 8, 2
    part = oracle.partition(m.key, 4)
    full = local_case(m, 0, l, K, D, seed=5, part=np.zeros(m.n_nodes, np.int32))
    gu = full["g"]
    ru = oracle.step(full["cfg"], gu, full["params"], full["nf"], full["ef"], None, None, want_v=True, want_e=True)
    # unpartitioned local ids are the global ids (one part, ascending)
    assert np.array_equal(gu["l2g"], np.arange(m.n_nodes))
    u_edge_of_global = np.empty(m.n_edges, np.int64)
    u_edge_of_global[gu["eperm"]] = np.arange(gu["n_edges"])
    for p in range(4):
        c = local_case(m, p, l, K, D, seed=5, part=part)
        g = c["g"]
        halo_ids = g["l2g"][g["n_owned"]:]
        H = np.stack([ru["v_all"][k][halo_ids] for k in range(K)])
        rp = oracle.step(c["cfg"], g, c["params"], c["nf"], c["ef"], H, None, want_e=True)
        assert _rel(rp["out"], ru["out"][g["l2g"][:g["n_owned"]]]) < 1e-12
        ue = u_edge_of_global[g["eperm"]]
        for k in range(K + 1):
            assert _rel(rp["e_all"][k], ru["e_all"][k][ue]) < 1e-12


def test_nocomm_keeps_interior_outputs():
    """The paper's NoComm variant (each part trained on its own nodes and the
    edges between them, no halo): an owned node whose receptive field (nodes
    within K in-edge hops) stays inside its part keeps the whole network's
    output exactly; the nodes next to the cut lose their cross-part messages
    and change."""
    from paper_2307_13592_amd.lockstep import nocomm_edges
    m = meshes.sector(4, 32, 6, 4, seed=7)
    K, l, D = 2, 8, 2
    part = oracle.partition(m.key, 4)
    full = local_case(m, 0, l, K, D, seed=5, part=np.zeros(m.n_nodes, np.int32))
    ru = oracle.step(full["cfg"], full["g"], full["params"], full["nf"], full["ef"], None, None)
    mn = meshes.Mesh(**{**m.__dict__})
    mn.send, mn.recv = nocomm_edges(m.send, m.recv, part)
    preds = [[] for _ in range(m.n_nodes)]
    for s_, r_ in zip(m.send, m.recv):
        preds[r_].append(s_)
    for p in (0, 1):
        c = local_case(mn, p, l, K, D, seed=5, part=part)
        g = c["g"]
        assert g["n_halo"] == 0
        rp = oracle.step(c["cfg"], g, c["params"], c["nf"], c["ef"], None, None)
        own = g["l2g"][:g["n_owned"]]
        inside = []
        for n in own:  # receptive field of n in the whole mesh, by breadth-first search
            field, front = {int(n)}, {int(n)}
            for _ in range(K):
                front = {int(s_) for r_ in front for s_ in preds[r_]} - field
                field |= front
            inside.append(all(part[x] == p for x in field))
        inside = np.asarray(inside)
        assert inside.any() and (~inside).any()
        assert _rel(rp["out"][inside], ru["out"][own[inside]]) < 1e-12
        assert np.abs(rp["out"][~inside] - ru["out"][own[~inside]]).max(axis=1).min() > 1e-6


def test_backward_is_linear_in_d_out():
    c = local_case(meshes.sector(3, 8, 4, 4, seed=2), 1, 8, 2, 3, seed=8)
    a = oracle.step(c["cfg"], c["g"], c["params"], c["nf"], c["ef"], c["halo"], c["d_out"])
    b = oracle.step(c["cfg"], c["g"], c["params"], c["nf"], c["ef"], c["halo"], 2.0 * c["d_out"])
    z = oracle.step(c["cfg"], c["g"], c["params"], c["nf"], c["ef"], c["halo"], 0.0 * c["d_out"])
    assert np.array_equal(b["d_params"], 2.0 * a["d_params"])
    assert np.array_equal(b["d_halo"], 2.0 * a["d_halo"])
    assert np.all(z["d_params"] == 0) and np.all(z["d_halo"] == 0)
    assert np.array_equal(a["out"], b["out"])


def test_scatter_sum_is_incidence_product():
    m = meshes.delaunay_box(4, 4, 4, seed=1)
    g = oracle.graph_build(m.send, m.recv, np.zeros(m.n_nodes, np.int32), m.n_nodes, 0)
    rng = np.random.default_rng(3)
    msg = rng.integers(-3, 4, (g["n_edges"], 5)).astype(np.int64)
    R = np.zeros((g["n_edges"], g["n_owned"]), np.int64)
    R[np.arange(g["n_edges"]), np.repeat(np.arange(g["n_owned"]), np.diff(g["row_ptr"]))] = 1
    assert np.array_equal(oracle.scatter_sum(g["row_ptr"], msg.astype(np.float64)), (R.T @ msg).astype(np.float64))
    # with messages = sender rows, the sum is the adjacency-count product A V
    V = rng.integers(-3, 4, (g["n_owned"], 3)).astype(np.int64)
    A = np.zeros((g["n_owned"], g["n_owned"]), np.int64)
    np.add.at(A, (np.repeat(np.arange(g["n_owned"]), np.diff(g["row_ptr"])), g["send"]), 1)
    assert np.array_equal(oracle.scatter_sum(g["row_ptr"], V[g["send"]].astype(np.float64)), (A @ V).astype(np.float64))


def test_layernorm_row_mean_is_mean_beta():
    """With gamma = 1 the encoder's LayerNorm rows average to mean(beta)."""
    c = local_case(meshes.hex_lattice(4), 0, 16, 1, 2, seed=2)
    P = c["params"].copy()
    for nm, sl in _segments(c["shapes"]):
        if nm == "enc_node.ln.gamma":
            P[sl] = 1.0
        if nm == "enc_node.ln.beta":
            beta = P[sl]
    r = oracle.step(c["cfg"], c["g"], P, c["nf"], c["ef"], None, None, want_v=True)
    v0 = r["v_all"][0]
    np.testing.assert_allclose(v0.mean(1), beta.mean(), rtol=0, atol=1e-13)
    assert np.all(((v0 - beta) ** 2).mean(1) <= 1.0)


def test_mse_grad_matches_autograd():
    rng = np.random.default_rng(4)
    out, tgt = rng.standard_normal((50, 5)), rng.standard_normal((50, 5))
    mask = rng.integers(0, 2, 50).astype(np.uint8)
    L, d = oracle.mse_grad(out, tgt, mask)
    o = torch.as_tensor(out).requires_grad_(True)
    mt = torch.as_tensor(mask.astype(bool))
    lt = ((o - torch.as_tensor(tgt))[mt] ** 2).mean()
    lt.backward()
    assert abs(L - lt.item()) < 1e-14
    assert _rel(d, o.grad.numpy()) < 1e-14
    L0, d0 = oracle.mse_grad(out, tgt, np.zeros(50, np.uint8))
    assert L0 == 0 and np.all(d0 == 0)


def test_sgd_step_against_torch_optimizer_and_closed_forms():
    """Algorithm 1's update: torch.optim.SGD (no momentum) on the same
    parameters and gradient gives the same values; on L = |theta - t|^2 / 2
    one step with lr = 1 lands exactly on t; lr = 0 changes nothing."""
    rng = np.random.default_rng(8)
    theta, grad = rng.standard_normal(1000), rng.standard_normal(1000)
    w = torch.nn.Parameter(torch.as_tensor(theta.copy()))
    opt = torch.optim.SGD([w], lr=0.037)
    w.grad = torch.as_tensor(grad.copy())
    opt.step()
    assert _rel(oracle.sgd_step(theta, grad, 0.037), w.detach().numpy()) < 1e-15
    t = rng.standard_normal(1000)
    half = np.round(theta * 64) / 64  # exact in binary: theta - (theta - t) has no rounding
    t = np.round(t * 64) / 64
    assert np.array_equal(oracle.sgd_step(half, half - t, 1.0), t)
    assert np.array_equal(oracle.sgd_step(theta, grad, 0.0), theta)


def test_rollout_update_special_cases():
    """q_{t+1} = p + q_t on the flow columns only: p = 0 changes nothing;
    p = -q zeroes the flow columns and leaves coordinates and type flags;
    two updates add."""
    rng = np.random.default_rng(9)
    nf = rng.standard_normal((40, 11))
    assert np.array_equal(oracle.rollout_update(nf, np.zeros((40, 5))), nf)
    z = oracle.rollout_update(nf, -nf[:, 3:8])
    assert not np.any(z[:, 3:8])
    assert np.array_equal(z[:, :3], nf[:, :3]) and np.array_equal(z[:, 8:], nf[:, 8:])
    p = np.round(rng.standard_normal((40, 5)) * 8) / 8
    q = np.round(nf * 8) / 8
    assert np.array_equal(oracle.rollout_update(oracle.rollout_update(q, p), p), oracle.rollout_update(q, 2 * p))
    with pytest.raises(ValueError):
        oracle.rollout_update(nf, np.zeros((40, 5)), col0=7)


def test_mse_global_shares_add_up_to_the_whole():
    """Algorithm 1's loss all-reduce: the parts' shares of the global mean
    add up to the mean over all rows, and their gradients are the rows of
    the whole loss's gradient (the single-call form is pinned to autograd
    above)."""
    rng = np.random.default_rng(6)
    out, tgt = rng.standard_normal((90, 5)), rng.standard_normal((90, 5))
    mask = rng.integers(0, 2, 90).astype(np.uint8)
    L, d = oracle.mse_grad(out, tgt, mask)
    cuts = [0, 20, 55, 90]
    rows = int(mask.sum())
    shares, grads = [], []
    for a, b in zip(cuts[:-1], cuts[1:]):
        l_p, d_p = oracle.mse_grad(out[a:b], tgt[a:b], mask[a:b], global_rows=rows)
        shares.append(l_p)
        grads.append(d_p)
    assert abs(sum(shares) - L) < 1e-14
    assert np.array_equal(np.concatenate(grads), d)


def test_norm_hand_case():
    """Normalize (Algorithm 1) on numbers worked by hand: rows 1 and 3 give
    mean 2 and population deviation 1, so 5 maps to 3 and 2 to 0; a column
    that never varies keeps deviation eps; no rows seen is the identity."""
    st = oracle.norm_accumulate(np.zeros(5), np.array([[1.0, 7.0], [3.0, 7.0]]))
    assert st.tolist() == [2.0, 4.0, 14.0, 10.0, 98.0]
    y = oracle.norm_apply(st, np.array([[5.0, 7.0], [2.0, 8.0]]), eps=0.5)
    assert y.tolist() == [[3.0, 0.0], [0.0, 2.0]]
    x = np.array([[-1.5, 2.0]])
    assert np.array_equal(oracle.norm_apply(np.zeros(5), x), x)


def test_norm_against_moments():
    """Statistics accumulated over three calls (one of them empty) equal one
    call over the concatenated rows, give numpy's mean and population
    variance of those rows, and standardise them to mean 0 and deviation 1
    per column; ragged row counts, 11 columns at different scales."""
    r = np.random.default_rng(12)
    parts = [r.normal(3.0, 0.5, (97, 11)) * np.arange(1, 12), np.zeros((0, 11)), r.normal(-2.0, 4.0, (1003, 11))]
    st = np.zeros(23)
    for x in parts:
        st = oracle.norm_accumulate(st, x)
    allx = np.concatenate(parts)
    one = oracle.norm_accumulate(np.zeros(23), allx)
    assert np.allclose(st, one, rtol=1e-13, atol=0)
    assert st[0] == len(allx)
    mean, var = st[1:12] / st[0], st[12:] / st[0] - (st[1:12] / st[0]) ** 2
    assert np.allclose(mean, allx.mean(0), rtol=1e-12) and np.allclose(var, allx.var(0), rtol=1e-10)
    y = oracle.norm_apply(st, allx)
    assert np.allclose(y.mean(0), 0, atol=1e-12) and np.allclose(y.std(0), 1, rtol=1e-10)
    with pytest.raises(ValueError):
        oracle.norm_accumulate(np.zeros(5), np.zeros((3, 4)))
    with pytest.raises(ValueError):
        oracle.norm_apply(np.zeros(5), np.zeros((3, 2)), eps=0.0)


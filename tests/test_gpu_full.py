"""GPU parity at the benchmark sizes, in the launch configuration bench.py
times (the whole partition in one step).

C4 runs with the first-Linear stash sized as bench.py sizes it (as many
blocks as the GPU's free memory holds: 13 of 15 on a 288 GB MI355X), and a
separate test checks that this plan gives bitwise the results of the plan
without the stash.  C5 runs with edge-stream checkpointing
(mgn_set_recompute).  C2 (100k-node Delaunay, fp32) is compared on every
output and every gradient tensor with the oracle's full-size run stored by
tests/golden/make_c2_reference.py.

Sampled outputs: an owned node's output after K blocks depends only on its
receptive field (tests/cone.py), so the oracle computes it on that
sub-graph.  With the loss gradient non-zero only on the sampled nodes, every
parameter gradient and every halo gradient of the full partition equals the
sub-graph's, which the oracle also computes.  Sampled nodes: local id 0 (the
slab's first theta layer at the hub and the inflow face, next to the halo)
and, except for C5, an interior node of the same layer (mid radius, mid
span).

Properties at full size: two runs agree bitwise; the backward pass is exactly
linear in the loss gradient; halo gradients outside the receptive field are
exactly zero.
"""
import gc
import os

import numpy as np
import pytest

import synth
import paper_2307_13592_amd as mgn
from paper_2307_13592_amd.runner import Session
from cone import cone, cone_digest
from parity import TOL, calibrate, compare, rel_err, run_oracle, say

pytestmark = pytest.mark.gpu


def _inputs(cfg):
    say(f"[full] {cfg.name}: building {cfg.note}")
    case = synth.make_case(cfg, region=True)
    m = case.mesh
    part = m.part if m.part is not None else np.zeros(m.n_nodes, np.int32)
    g = mgn.mgn_graph_build(m.send, m.recv, part, m.n_nodes, cfg.part)
    loc = case.local_inputs(g["l2g"], g["eperm"], g["n_owned"], g["n_halo"])
    say(f"[full] {cfg.name}: owned {g['n_owned']}, halo {g['n_halo']}, edges {g['n_edges']}")
    return case, g, loc


def _free(s):
    import torch
    s.close()
    gc.collect()
    torch.cuda.empty_cache()


# edge-stream checkpoint interval per configuration: C5's stash-all workspace
# (~430 GB of edge latents alone) does not fit one GPU
RECOMPUTE = {"C5": -1}
# first-Linear stash per configuration, as bench.py runs it (-1: as many
# blocks as the free memory holds)
H1_STASH = {"C4": -1}


def _session(name, cfg, case, g, loc, h1_stash=None):
    s = Session(cfg.latent, cfg.K, cfg.depth, cfg.precision, g, loc["node_feat"], loc["edge_feat"], loc["halo"],
                case.params, recompute=RECOMPUTE.get(name, 0),
                h1_stash=H1_STASH.get(name, 0) if h1_stash is None else h1_stash)
    say(f"[full] {name}: workspace {s.ws_bytes / 2**30:.1f} GiB, first-Linear stash {s.h1_stash} of {cfg.K} blocks")
    return s


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["C3", "C4", "C5"])
def test_sampled_outputs_and_gradients(name):
    cfg = synth.CONFIGS[name]
    case, g, loc = _inputs(cfg)
    no, l, K, D = g["n_owned"], cfg.latent, cfg.K, cfg.depth
    n_r, n_z = (50, 500) if name == "C3" else (100, 500)
    r_mid, z_mid = n_r // 2, 250
    # C5 (l=256, D=3): node 0 alone keeps the CPU oracle's share to minutes
    centers = np.array([0] if name == "C5" else [0, r_mid * n_z + z_mid])
    d_out = np.zeros((no, 5), np.float32)
    d_out[centers] = np.random.default_rng([cfg.seed, 5]).standard_normal((centers.size, 5)).astype(np.float32)
    s = _session(name, cfg, case, g, loc)
    if name == "C4":
        assert s.h1_stash > 0, "the benchmarked C4 plan stashes h_1"
    try:
        say(f"[full] {name}: GPU step")
        out = s.forward().cpu().numpy()
        dp, dh = s.backward(d_out)
        dp, dh = dp.cpu().numpy().copy(), dh.cpu().numpy().copy()
    finally:
        _free(s)
    c = cone(g, centers, K)
    say(f"[full] {name}: receptive field {c['n_owned']} owned + {c['n_halo']} halo nodes, {c['n_edges']} edges")
    sub = dict(g=c, shapes=case.shapes, params=case.params, nf=loc["node_feat"][c["owned"]],
               ef=loc["edge_feat"][c["edges"]], halo=loc["halo"][:, c["halo"]],
               d_out=d_out[c["owned"]])
    ref = run_oracle(sub, l, K, D, bf16=cfg.precision == "bf16")
    say(f"[full] {name}: oracle done")
    cal = calibrate(sub, l, K, D, cfg.precision, runs=4)
    say(f"[full] {name}: calibration done")
    # the oracle's own movement under float32-level input noise, eight runs
    # on this cone, written by tests/golden/make_cone_sensitivity.py (oracle
    # only): K = 15 blocks amplify such noise into movements of 0.1-0.7 in
    # some bf16 gradient tensors (ReLU flips), and eight runs sample that
    # spread (three missed the largest movement of block 10's node Linear at
    # C5, 0.22, which the oracle alone reaches in one of eight)
    fx = np.load(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                              f"cone_sensitivity_{name}.npz"))
    assert str(fx["digest"]) == cone_digest(c, sub, case.params), "the stored sensitivity belongs to other inputs"
    assert list(fx["names"]) == [s[0] for s in case.shapes]
    sens = {"d_params": fx["sens_d_params"], "d_halo": float(fx["sens_d_halo"])}
    # outputs at the sampled nodes only
    e_out = rel_err(out[centers], ref["out"][c["centers_sub"]])
    ref_c = dict(ref)
    ref_c["out"] = ref["out"][c["centers_sub"]]
    bad = compare(f"{name} sampled", cfg.precision, case.shapes, (out[centers], dp, dh), ref_c, cal,
                  halo_sel=c["halo"], sens=sens)
    assert e_out <= TOL[cfg.precision]
    assert not bad, bad
    outside = np.setdiff1d(np.arange(g["n_halo"]), c["halo"])
    assert not np.any(dh[:, outside]), "halo gradient outside the receptive field must be zero"


@pytest.mark.parametrize("name", ["C2", "C3", "C4"])
def test_full_size_determinism_and_linearity(name):
    cfg = synth.CONFIGS[name]
    case, g, loc = _inputs(cfg)
    d_out = np.random.default_rng([cfg.seed, 6]).standard_normal((g["n_owned"], 5)).astype(np.float32)
    s = _session(name, cfg, case, g, loc)
    try:
        say(f"[full] {name}: run 1")
        o1 = s.forward().cpu().numpy().copy()
        p1, h1 = (x.cpu().numpy().copy() if x is not None else None for x in s.backward(d_out))
        say(f"[full] {name}: run 2")
        o2 = s.forward().cpu().numpy().copy()
        p2, h2 = (x.cpu().numpy().copy() if x is not None else None for x in s.backward(d_out))
        assert np.array_equal(o1, o2) and np.array_equal(p1, p2)
        if h1 is not None:
            assert np.array_equal(h1, h2)
        say(f"[full] {name}: doubled loss gradient")
        p3, h3 = (x.cpu().numpy().copy() if x is not None else None for x in s.backward(2.0 * d_out))
        assert np.array_equal(p3, 2.0 * p1)
        if h1 is not None:
            assert np.array_equal(h3, 2.0 * h1)
        assert np.all(np.isfinite(o1)) and np.all(np.isfinite(p1))
    finally:
        _free(s)




def _step(s, d_out):
    out = s.forward().cpu().numpy().copy()
    dp, dh = s.backward(d_out)
    return out, dp.cpu().numpy().copy(), None if dh is None else dh.cpu().numpy().copy()


def test_c4_stash_plan_bitwise():
    """The benchmarked C4 plan (first-Linear stash for as many blocks as fit,
    their forwards sharing one node-projection slot) gives bitwise the
    outputs, parameter gradients and halo gradients of the plan without the
    stash, at full size."""
    cfg = synth.CONFIGS["C4"]
    case, g, loc = _inputs(cfg)
    d_out = np.random.default_rng([cfg.seed, 8]).standard_normal((g["n_owned"], 5)).astype(np.float32)
    s = _session("C4", cfg, case, g, loc, h1_stash=-1)
    n_st = s.h1_stash
    try:
        assert 0 < n_st <= cfg.K
        say(f"[full] C4: step with {n_st} stashed blocks")
        a = _step(s, d_out)
    finally:
        _free(s)
    s = _session("C4", cfg, case, g, loc, h1_stash=0)
    try:
        say("[full] C4: step without the stash")
        b = _step(s, d_out)
    finally:
        _free(s)
    for nm, x, y in zip(("outputs", "parameter gradients", "halo gradients"), a, b):
        assert np.array_equal(x, y), f"{nm} differ ({n_st} stashed blocks): {rel_err(x, y):.2e}"


def test_c2_against_oracle():
    """C2 at full size (100k nodes, 1.55M edges, l=128, K=15, fp32): every
    output and every gradient tensor against the oracle's float64 run stored
    in tests/golden/c2_reference.npz (written by
    tests/golden/make_c2_reference.py, which calls only the oracle and the
    input generator); the loss gradient is the fixture's N(0,1) draw.
    Outputs within 1e-4; each gradient tensor within bound_of(): 1e-4, or
    twice the oracle's own movement under float32-level input noise (stored
    in the fixture) when that is larger, capped at 5e-4 unless the oracle's
    movement alone reaches half of it."""
    import os
    import sys
    from parity import bound_of, log_bounds, segments
    sys.path.insert(0, os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden"))
    import make_c2_reference as ref_script
    fx = np.load(ref_script.OUT)
    cfg = synth.CONFIGS["C2"]
    case, g, loc = _inputs(cfg)
    d_out = np.random.default_rng([cfg.seed, 7]).standard_normal((g["n_owned"], 5)).astype(np.float32)
    # the library's local graph and the inputs are the ones the oracle ran on
    assert ref_script.input_digest(g, loc, case.params, d_out) == str(fx["digest"])
    s = _session("C2", cfg, case, g, loc)
    try:
        say("[full] C2: GPU step")
        out, dp, _ = _step(s, d_out)
    finally:
        _free(s)
    rows, bad = [], []
    e = rel_err(out, fx["out"])
    rows.append(("out", e, None, None, TOL["fp32"]))
    if e > TOL["fp32"]:
        bad.append(("out", e))
    ref = fx["d_params"].astype(np.float64)
    for i, (nm, sl) in enumerate(segments(case.shapes)):
        e = rel_err(dp[sl], ref[sl])
        sens = float(fx["sens_d_params"][i])
        b = bound_of("fp32", None, sens)
        rows.append((nm, e, None, sens, b))
        if e > b:
            bad.append((nm, e, b))
    log_bounds("C2 full size", "fp32", rows)
    w = max(rows, key=lambda r: r[1] / r[4])
    say(f"  C2 full size: out {rows[0][1]:.2e}; tightest {w[0]} {w[1]:.2e} (bound {w[4]:.2e})")
    assert not bad, bad

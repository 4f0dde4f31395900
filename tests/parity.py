"""Shared helpers of the GPU parity tests: run one case through libmgn's C ABI
and through the oracle on the same seeded fp32 inputs, compare per tensor."""
from __future__ import annotations

import sys

import numpy as np

import oracle
import synth
import paper_2307_13592_amd as mgn
from paper_2307_13592_amd.runner import Session

TOL = {"fp32": 1e-4, "bf16": 2e-2}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def rel_err(got, ref) -> float:
    """max |got - ref| / max |ref| (absolute when ref is all zero)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    if ref.size == 0:
        return 0.0
    den = np.abs(ref).max()
    d = np.abs(got - ref).max()
    return float(d / den) if den > 0 else float(d)


def segments(shapes):
    off = 0
    for name, _, shape in shapes:
        n = int(np.prod(shape))
        yield name, slice(off, off + n)
        off += n


def local_inputs(mesh, p, latent, K, depth, seed, part=None):
    """libmgn-built local graph and fp32 inputs (as numpy)."""
    if part is None:
        part = mesh.part if mesh.part is not None else mgn.mgn_partition_slabs(mesh.key, mesh.nparts)
    g = mgn.mgn_graph_build(mesh.send, mesh.recv, part, mesh.n_nodes, p)
    shapes = synth.param_shapes(latent, K, depth)
    params = synth.init_params(shapes, seed)
    nf = synth.node_features(mesh, seed)[g["l2g"][:g["n_owned"]]]
    ef = synth.edge_features(mesh)[g["eperm"]]
    halo = synth.halo_latents(K, g["n_halo"], latent, seed)
    d_out = np.random.default_rng([seed, 99]).standard_normal((g["n_owned"], 5)).astype(np.float32)
    return dict(g=g, shapes=shapes, params=params, nf=nf, ef=ef, halo=halo, d_out=d_out, part=part)


def run_gpu(c, latent, K, depth, prec, d_out=None):
    s = Session(latent, K, depth, prec, c["g"], c["nf"], c["ef"], c["halo"], c["params"])
    try:
        out = s.forward().cpu().numpy().copy()
        dp, dh = s.backward(c["d_out"] if d_out is None else d_out)
        dp = dp.cpu().numpy().copy()
        dh = dh.cpu().numpy().copy() if dh is not None else np.zeros((K, 0, latent), np.float32)
    finally:
        s.close()
    return out, dp, dh


def run_oracle(c, latent, K, depth, d_out=None, g=None, nf=None, ef=None, halo=None, bf16=False):
    """The oracle on the same fp32 inputs; bf16=True selects its mixed-precision
    mode (bfloat16 operands at the same points as the bf16 kernels)."""
    cfg = oracle.ModelCfg(latent, K, depth, bf16=bf16)
    g = c["g"] if g is None else g
    r = oracle.step(cfg, g, c["params"].astype(np.float64),
                    (c["nf"] if nf is None else nf).astype(np.float64),
                    (c["ef"] if ef is None else ef).astype(np.float64),
                    (c["halo"] if halo is None else halo).astype(np.float64) if g["n_halo"] else None,
                    (c["d_out"] if d_out is None else d_out).astype(np.float64))
    return r


def compare(name, prec, shapes, gpu, ref, halo_sel=None):
    """Per-tensor max relative error; returns the list of failures."""
    out, dp, dh = gpu
    tol = TOL[prec]
    bad = []
    e = rel_err(out, ref["out"])
    worst = ("out", e)
    if e > tol:
        bad.append(("out", e))
    for nm, sl in segments(shapes):
        e = rel_err(dp[sl], ref["d_params"][sl])
        if e > worst[1]:
            worst = (nm, e)
        if e > tol:
            bad.append((nm, e))
    if ref["d_halo"].size:
        e = rel_err(dh if halo_sel is None else dh[:, halo_sel], ref["d_halo"])
        if e > worst[1]:
            worst = ("d_halo", e)
        if e > tol:
            bad.append(("d_halo", e))
    say(f"  {name}: worst {worst[0]} {worst[1]:.2e} (tol {tol:g})")
    return bad

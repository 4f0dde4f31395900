"""Writes tests/golden/cone_sensitivity_<config>.npz for the full-size sampled
parity test of C3, C4 and C5: how far the oracle's own parameter and halo
gradients on the test's receptive-field cone move, tensor by tensor, when
the cone's node features, edge features and halo latents are perturbed at the
float32 level (synth.perturbed, SENS_RUNS runs against the unperturbed run).
Fifteen blocks amplify such noise into movements of tens of percent in some
bf16 gradient tensors (ReLU units within rounding distance of zero); the test
widens a tensor's bound to twice the larger of this movement and that of an
independent float32 implementation, and reads the movement from here because
eight oracle runs on a cone take several minutes.

Only the seeded input generator (synth), the receptive-field extraction
(tests/cone.py) and the oracle are called: the graph is built by the oracle's
own graph_build, the cone and the loss gradient are the test's.  Run from the
repository root:

    python tests/golden/make_cone_sensitivity.py C3 C4 C5

(about a minute per oracle run and configuration on 8 host cores; the oracle
uses every OpenMP thread)."""
from __future__ import annotations

import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)
sys.path.insert(0, os.path.dirname(HERE))

import oracle  # noqa: E402
import synth  # noqa: E402
from cone import cone, cone_digest  # noqa: E402

SENS_RUNS = 8
REL = 2.0 ** -20


def out_path(name: str) -> str:
    return os.path.join(HERE, f"cone_sensitivity_{name}.npz")


def cone_inputs(name: str):
    """The sampled test's cone and inputs, in the oracle's local order."""
    cfg = synth.CONFIGS[name]
    case = synth.make_case(cfg, region=True)
    m = case.mesh
    part = m.part if m.part is not None else np.zeros(m.n_nodes, np.int32)
    g = oracle.graph_build(m.send, m.recv, part, m.n_nodes, cfg.part)
    loc = case.local_inputs(g["l2g"], g["eperm"], g["n_owned"], g["n_halo"])
    no = g["n_owned"]
    n_r, n_z = (50, 500) if name == "C3" else (100, 500)
    r_mid, z_mid = n_r // 2, 250
    centers = np.array([0] if name == "C5" else [0, r_mid * n_z + z_mid])
    d_out = np.zeros((no, 5), np.float32)
    d_out[centers] = np.random.default_rng([cfg.seed, 5]).standard_normal((centers.size, 5)).astype(np.float32)
    c = cone(g, centers, cfg.K)
    sub = dict(nf=loc["node_feat"][c["owned"]], ef=loc["edge_feat"][c["edges"]], halo=loc["halo"][:, c["halo"]],
               d_out=d_out[c["owned"]])
    return cfg, case, c, sub


def rel(a, ref) -> float:
    den = np.abs(ref).max() if ref.size else 0.0
    d = np.abs(a - ref).max() if ref.size else 0.0
    return float(d / den) if den > 0 else float(d)


def make(name: str):
    t = time.time()
    cfg, case, c, sub = cone_inputs(name)
    print(f"{name}: cone {c['n_owned']} owned + {c['n_halo']} halo nodes, {c['n_edges']} edges; "
          f"inputs {time.time() - t:.1f}s", flush=True)
    ocfg = oracle.ModelCfg(cfg.latent, cfg.K, cfg.depth, bf16=cfg.precision == "bf16")
    params = case.params.astype(np.float64)

    def run(nf, ef, halo):
        t = time.time()
        r = oracle.step(ocfg, c, params, nf.astype(np.float64), ef.astype(np.float64),
                        halo.astype(np.float64) if c["n_halo"] else None, sub["d_out"].astype(np.float64))
        print(f"  oracle step {time.time() - t:.1f}s", flush=True)
        return r

    ref = run(sub["nf"], sub["ef"], sub["halo"])
    sens = np.zeros(len(case.shapes))
    sens_halo = 0.0
    for i in range(1, SENS_RUNS + 1):
        nf, ef, halo = synth.perturbed((sub["nf"], sub["ef"], sub["halo"]), i, REL)
        r = run(nf, ef, halo)
        off = 0
        for k, (_, _, shape) in enumerate(case.shapes):
            n = int(np.prod(shape))
            sens[k] = max(sens[k], rel(r["d_params"][off:off + n], ref["d_params"][off:off + n]))
            off += n
        if ref["d_halo"].size:
            sens_halo = max(sens_halo, rel(r["d_halo"], ref["d_halo"]))
    np.savez(out_path(name), sens_d_params=sens, sens_d_halo=sens_halo, sens_runs=SENS_RUNS, rel=REL,
             names=np.array([s[0] for s in case.shapes]), digest=cone_digest(c, sub, case.params))
    print(f"wrote {out_path(name)}", flush=True)


if __name__ == "__main__":
    for nm in sys.argv[1:] or ["C3", "C4", "C5"]:
        make(nm)

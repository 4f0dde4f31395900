"""Writes tests/golden/c2_reference.npz: the oracle's outputs and parameter
gradients for the whole 100k-node Delaunay workload (latent 128, 15 blocks,
2-layer MLPs, float32 inputs, float64 arithmetic), for the GPU parity test of
that workload, and how far the oracle's own gradients move, tensor by tensor,
when its node and edge features are perturbed at the float32 level
(synth.perturbed, SENS_RUNS runs): the widening of the parity bound that
ReLU units sitting within rounding distance of zero justify, shown by the
oracle alone.

Only the seeded input generator (synth) and the oracle are called: the graph
is built by the oracle's own graph_build, the loss gradient is N(0,1) from a
numpy generator seeded with (config seed, 7).  Run from the repository root:

    python tests/golden/make_c2_reference.py

(about 5 minutes per oracle run on 16 host cores, 1 + SENS_RUNS runs; the
oracle uses every OpenMP thread).  With --extend, an existing fixture of the
same inputs keeps its reference run and only the missing perturbed runs are
made (their movement is merged by taking the larger)."""
from __future__ import annotations

import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import synth  # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c2_reference.npz")
SENS_RUNS = 6


def c2_inputs():
    """C2's seeded inputs in the oracle's local order (one partition, no halo)."""
    cfg = synth.CONFIGS["C2"]
    case = synth.make_case(cfg, region=True)
    m = case.mesh
    g = oracle.graph_build(m.send, m.recv, np.zeros(m.n_nodes, np.int32), m.n_nodes, 0)
    loc = case.local_inputs(g["l2g"], g["eperm"], g["n_owned"], g["n_halo"])
    d_out = np.random.default_rng([cfg.seed, 7]).standard_normal((g["n_owned"], 5)).astype(np.float32)
    return cfg, case, g, loc, d_out


def input_digest(g, loc, params, d_out) -> str:
    """sha256 over the local graph and every input array, in order, so a
    reader can tell the fixture belongs to the inputs it regenerates."""
    import hashlib
    h = hashlib.sha256()
    for a in (g["row_ptr"], g["send"], g["l2g"], g["eperm"], loc["node_feat"], loc["edge_feat"], params, d_out):
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


def tensor_rel_err(a, ref, shapes) -> np.ndarray:
    """Per parameter tensor (flat layout order): max |a - ref| / max |ref|."""
    out, off = [], 0
    for _, _, shape in shapes:
        n = int(np.prod(shape))
        den = np.abs(ref[off:off + n]).max()
        d = np.abs(a[off:off + n] - ref[off:off + n]).max()
        out.append(d / den if den > 0 else d)
        off += n
    return np.array(out)


def main():
    t = time.time()
    cfg, case, g, loc, d_out = c2_inputs()
    print(f"C2: {g['n_owned']} nodes, {g['n_edges']} edges; inputs {time.time() - t:.1f}s", flush=True)
    ocfg = oracle.ModelCfg(cfg.latent, cfg.K, cfg.depth)
    params = case.params.astype(np.float64)
    digest = input_digest(g, loc, case.params, d_out)

    def run(nf, ef):
        t = time.time()
        r = oracle.step(ocfg, g, params, nf, ef, None, d_out.astype(np.float64))
        print(f"oracle step {time.time() - t:.1f}s", flush=True)
        return r

    first = 1
    if "--extend" in sys.argv and os.path.exists(OUT):
        old = np.load(OUT)
        assert str(old["digest"]) == digest, "the stored fixture belongs to other inputs"
        # the stored float32 copy of the reference, as the GPU test reads it
        r = {"out": old["out"].astype(np.float64), "d_params": old["d_params"].astype(np.float64)}
        sens, sens_out, first = old["sens_d_params"].copy(), float(old["sens_out"]), int(old["sens_runs"]) + 1
    else:
        r = run(loc["node_feat"].astype(np.float64), loc["edge_feat"].astype(np.float64))
        sens = np.zeros(len(case.shapes))
        sens_out = 0.0
    for i in range(first, SENS_RUNS + 1):
        nf, ef = synth.perturbed((loc["node_feat"], loc["edge_feat"]), i)
        rp = run(nf, ef)
        sens = np.maximum(sens, tensor_rel_err(rp["d_params"], r["d_params"], case.shapes))
        sens_out = max(sens_out, float(np.abs(rp["out"] - r["out"]).max() / np.abs(r["out"]).max()))
    np.savez(OUT, out=r["out"].astype(np.float32), d_params=r["d_params"].astype(np.float32),
             sens_d_params=sens, sens_out=sens_out, sens_runs=SENS_RUNS, n_owned=g["n_owned"],
             n_edges=g["n_edges"], digest=digest)
    print(f"wrote {OUT}", flush=True)


if __name__ == "__main__":
    main()

"""The stored oracle fixtures under tests/golden/ against the configurations
they were written for (CPU): the full-size tests on the GPU machine refuse a
fixture whose cone digest differs, and these checks catch a change of the
input generator or of the parameter layout here, before a GPU run."""
import os

import numpy as np
import pytest

import oracle
import synth
from cone import cone, cone_digest

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


@pytest.mark.parametrize("name", ["C3", "C4", "C5"])
def test_cone_sensitivity_layout(name):
    cfg = synth.CONFIGS[name]
    fx = np.load(os.path.join(GOLDEN, f"cone_sensitivity_{name}.npz"))
    shapes = synth.param_shapes(cfg.latent, cfg.K, cfg.depth)
    assert list(fx["names"]) == [s[0] for s in shapes]
    sens = fx["sens_d_params"]
    assert sens.shape == (len(shapes),)
    assert np.all(np.isfinite(sens)) and np.all(sens >= 0)
    assert np.isfinite(float(fx["sens_d_halo"])) and float(fx["sens_d_halo"]) >= 0
    assert int(fx["sens_runs"]) == 8 and float(fx["rel"]) == 2.0 ** -20
    if cfg.precision == "fp32":
        # float64 oracle under 2^-20 input noise: small movements, except
        # near rounding-distance ReLU units, which the bound then absorbs
        assert np.median(sens) < 1e-4
    else:
        # the bf16 mode rounds at the kernels' points: 15 blocks amplify
        # the noise into movements of several percent in most tensors
        assert 1e-3 < np.median(sens) < 1.0


def test_cone_sensitivity_digest_c3():
    """The C3 fixture was written for exactly the cone and inputs the
    full-size test builds (the oracle's own graph build here; the GPU test
    uses the library's, which matches it bit for bit)."""
    cfg = synth.CONFIGS["C3"]
    case = synth.make_case(cfg, region=True)
    m = case.mesh
    g = oracle.graph_build(m.send, m.recv, m.part, m.n_nodes, cfg.part)
    loc = case.local_inputs(g["l2g"], g["eperm"], g["n_owned"], g["n_halo"])
    no = g["n_owned"]
    centers = np.array([0, 25 * 500 + 250])
    d_out = np.zeros((no, 5), np.float32)
    d_out[centers] = np.random.default_rng([cfg.seed, 5]).standard_normal((centers.size, 5)).astype(np.float32)
    c = cone(g, centers, cfg.K)
    sub = dict(nf=loc["node_feat"][c["owned"]], ef=loc["edge_feat"][c["edges"]], halo=loc["halo"][:, c["halo"]],
               d_out=d_out[c["owned"]])
    fx = np.load(os.path.join(GOLDEN, "cone_sensitivity_C3.npz"))
    assert cone_digest(c, sub, case.params) == str(fx["digest"])

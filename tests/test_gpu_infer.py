"""Forward-only (inference) plan and next-step rollout on the GPU: the
inference plan's outputs are bitwise those of the training plan (same
kernels and arithmetic, less memory) and it refuses a backward; a
three-step rollout (each prediction fed back into the flow columns,
q <- q + p) matches the oracle doing the same, step by step, to the
precision's output tolerance."""
import numpy as np
import pytest

import oracle
from synth import meshes
import paper_2307_13592_amd as mgn
from paper_2307_13592_amd.runner import Session
from parity import TOL, local_inputs, rel_err, run_oracle, say

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("prec,l,D", [("fp32", 128, 2), ("bf16", 128, 2), ("bf16", 256, 3), ("bf16", 64, 2)])
def test_inference_plan_is_bitwise_the_training_forward(prec, l, D):
    say(f"[infer] sector 6x16x10 p1 l={l} D={D} {prec}")
    c = local_inputs(meshes.sector(6, 16, 10, 4, seed=7), 1, l, 3, D, 4)
    outs, sizes = [], []
    for inference in (False, True):
        s = Session(l, 3, D, prec, c["g"], c["nf"], c["ef"], c["halo"], c["params"], inference=inference)
        try:
            outs.append(s.forward().cpu().numpy().copy())
            sizes.append(s.ws_bytes)
            if inference:
                import torch
                with pytest.raises(mgn.MgnError) as e:
                    mgn.mgn_backward(s.model, torch.zeros_like(s.out), torch.empty(s.n_params, device=s.device))
                assert e.value.status == mgn.MGN_E_STATE
        finally:
            s.close()
    say(f"  workspace {sizes[0]} -> {sizes[1]} bytes")
    assert np.array_equal(outs[0], outs[1])
    assert sizes[1] < sizes[0]


@pytest.mark.parametrize("prec", ["fp32", "bf16"])
def test_rollout_matches_oracle(prec):
    """Whole mesh (no halo), three next-step predictions."""
    say(f"[infer] rollout, delaunay 8x7x6, {prec}")
    mesh = meshes.delaunay_box(8, 7, 6, seed=3)
    c = local_inputs(mesh, 0, 128, 2, 2, 6, part=np.zeros(mesh.n_nodes, np.int32))
    s = Session(128, 2, 2, prec, c["g"], c["nf"], c["ef"], c["halo"], c["params"], inference=True)
    try:
        gpu = [o.cpu().numpy() for o in s.rollout(3)]
        nf_end = s.node_feat.cpu().numpy()
    finally:
        s.close()
    nf = c["nf"].astype(np.float64)
    for t in range(3):
        ref = run_oracle(c, 128, 2, 2, nf=nf, bf16=prec == "bf16")["out"]
        e = rel_err(gpu[t], ref)
        say(f"  step {t}: out {e:.2e}")
        assert e <= TOL[prec]
        nf = oracle.rollout_update(nf, ref)
    assert rel_err(nf_end, nf) <= TOL[prec]

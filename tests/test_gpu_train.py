"""Algorithm 1's training loop on the GPU: the parameter update
(theta <- theta - lr * grad, mgn_sgd_step) against the oracle's, the
refreshed packed weights by a forward pass against the oracle's network at
the updated parameters, three full training steps (forward, loss gradient,
backward, update) against the oracle's, and the lockstep parts staying in
step (identical parameters) after an update with their summed gradient."""
import numpy as np
import pytest
import torch

import oracle
from synth import meshes
import paper_2307_13592_amd as mgn
from paper_2307_13592_amd.runner import Session
from parity import TOL, local_inputs, rel_err, run_oracle, say

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("prec", ["fp32", "bf16"])
def test_sgd_step_matches_oracle(prec):
    say(f"[train] sgd step {prec}")
    c = local_inputs(meshes.sector(6, 16, 10, 4, seed=7), 1, 64, 2, 2, 3)
    s = Session(64, 2, 2, prec, c["g"], c["nf"], c["ef"], c["halo"], c["params"])
    try:
        grad = np.random.default_rng(12).standard_normal(s.n_params).astype(np.float32)
        lr = float(np.float32(0.01))  # the learning rate the kernel gets, exactly
        s.sgd(lr, torch.as_tensor(grad).to(s.device))
        got = mgn.mgn_get_params(s.model).astype(np.float64)
        want = oracle.sgd_step(c["params"], grad, lr)
        # one rounding of the exact value: within half a float32 ulp (plus
        # the float64 rounding of the oracle's own value)
        ulp = np.spacing(np.abs(want).astype(np.float32)).astype(np.float64)
        bad = np.abs(got - want) > 0.5 * ulp * (1 + 1e-6)
        assert not bad.any(), (int(bad.sum()), got[bad][:4], want[bad][:4])
        # the kernels use the refreshed packed weights
        out = s.forward().cpu().numpy()
        c2 = dict(c, params=want.astype(np.float32))
        ref = run_oracle(c2, 64, 2, 2, bf16=prec == "bf16")
        e = rel_err(out, ref["out"])
        say(f"  forward after the update: out {e:.2e}")
        assert e <= TOL[prec]
    finally:
        s.close()


def test_training_steps_match_oracle():
    """Three steps of forward, MSE gradient, backward and update in fp32:
    losses and final parameters against the oracle doing the same."""
    say("[train] three fp32 training steps")
    c = local_inputs(meshes.sector(6, 16, 10, 4, seed=7), 1, 64, 2, 2, 5)
    target = np.random.default_rng(21).standard_normal((c["g"]["n_owned"], 5)).astype(np.float32)
    lr = 0.01
    s = Session(64, 2, 2, "fp32", c["g"], c["nf"], c["ef"], c["halo"], c["params"])
    try:
        tgt = torch.as_tensor(target).to(s.device)
        gpu_losses = []
        for _ in range(3):
            s.forward()
            loss, d_out = s.mse(tgt)
            s.backward(d_out)
            s.sgd(lr)
            gpu_losses.append(float(loss[0].item()))
        gpu_params = mgn.mgn_get_params(s.model)
    finally:
        s.close()
    theta = c["params"].astype(np.float64)
    ref_losses = []
    for _ in range(3):
        r = run_oracle(dict(c, params=theta), 64, 2, 2, d_out=np.zeros_like(target))
        L, d_out = oracle.mse_grad(r["out"], target)
        r = run_oracle(dict(c, params=theta), 64, 2, 2, d_out=d_out)
        theta = oracle.sgd_step(theta, r["d_params"], lr)
        ref_losses.append(L)
    say(f"  losses gpu {gpu_losses} oracle {ref_losses}")
    assert ref_losses[-1] < ref_losses[0]
    for a, b in zip(gpu_losses, ref_losses):
        assert abs(a - b) / b <= TOL["fp32"]
    e = rel_err(gpu_params, theta)
    say(f"  parameters after 3 steps: {e:.2e}")
    assert e <= TOL["fp32"]


def test_lockstep_parts_stay_identical():
    """A lockstep training step with Algorithm 1's global loss: the parts'
    loss shares add up to the whole network's loss (oracle, bf16 mode), and
    after the update every part holds the same parameters."""
    from test_gpu_lockstep import _lockstep_session
    say("[train] lockstep update, bf16")
    mesh = meshes.sector(5, 12, 9, 4, seed=2)
    ls, whole, own = _lockstep_session(mesh, 4, 128, 2, 2, "bf16", 5)
    target = np.random.default_rng(31).standard_normal((mesh.n_nodes, 5)).astype(np.float32)
    try:
        ls.forward()
        shares, d_outs = ls.mse([torch.as_tensor(target[o]).to(ls.device) for o in own])
        gpu_loss = sum(float(x.item()) for x in shares)
        ref_out = run_oracle(whole, 128, 2, 2, bf16=True)["out"]
        ref_loss, _ = oracle.mse_grad(ref_out, target)
        say(f"  global loss gpu {gpu_loss:.6f} oracle {ref_loss:.6f}")
        assert abs(gpu_loss - ref_loss) / ref_loss <= TOL["bf16"]
        ls.backward(d_outs)
        ls.sgd(0.02)
        ps = [mgn.mgn_get_params(s.model) for s in ls.sessions]
        assert not np.array_equal(ps[0], whole["params"])
        for p in ps[1:]:
            assert np.array_equal(p, ps[0])
    finally:
        ls.close()

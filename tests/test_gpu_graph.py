"""The training step captured into a HIP graph (through torch.cuda.graph on
the library's stream argument) and replayed: the step makes no allocation,
synchronisation or memset, so every replay must give bitwise the eager
step's outputs, parameter gradients and halo gradients.  Between replays the
program does its own eager work (it overwrites the outputs) and
synchronises; each replay is checked."""
import numpy as np
import pytest
import torch

from synth import meshes
from paper_2307_13592_amd.runner import Session
from parity import local_inputs, say

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("prec,recompute", [("fp32", 0), ("bf16", 0), ("bf16", 2)])
def test_graph_replays_equal_eager_step(prec, recompute):
    say(f"[graph] sector 6x16x10 p1 l=128 K=3 {prec} recompute={recompute}")
    c = local_inputs(meshes.sector(6, 16, 10, 4, seed=7), 1, 128, 3, 2, 3)
    target = np.random.default_rng(5).standard_normal((c["g"]["n_owned"], 5)).astype(np.float32)
    s = Session(128, 3, 2, prec, c["g"], c["nf"], c["ef"], c["halo"], c["params"], recompute=recompute,
                chunk_edges=1000 if recompute else 0)
    try:
        tgt = torch.as_tensor(target).to(s.device)

        def step():
            s.forward()
            _, d_out = s.mse(tgt)
            s.backward(d_out)

        step()
        torch.cuda.synchronize()
        ref = [x.clone() for x in (s.out, s.d_params, s.d_halo)]
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step()  # warm-up on the capture stream
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step()
        for i in range(3):
            s.out.fill_(3.0)
            s.d_params.fill_(-7.0)
            s.d_halo.zero_()
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            for x, y in zip((s.out, s.d_params, s.d_halo), ref):
                assert torch.equal(x, y), f"replay {i} differs"
        say("  3 replays equal the eager step")
        del g
    finally:
        s.close()

"""mgn_forward_noalloc (the forward with the library's static per-GPU
workspace, for callers that cannot allocate) against mgn_forward with a
caller workspace, through the C ABI: outputs bitwise equal on two calls in a
row, the second on a smaller graph; an oversized graph is refused before
anything runs; a backward right after it matches the one after mgn_forward."""
import numpy as np
import pytest
import torch

from synth import meshes
import paper_2307_13592_amd as mgn
from paper_2307_13592_amd.runner import Session
from parity import local_inputs, say

pytestmark = pytest.mark.gpu


def _noalloc_out(s):
    out = torch.full_like(s.out, float("nan"))
    mgn.mgn_forward_noalloc(s.model, s.gs, s.node_feat, s.edge_feat, s.halo, out)
    return out.cpu().numpy()


@pytest.mark.parametrize("prec,l,D,infer", [("fp32", 64, 2, False), ("bf16", 128, 2, True), ("bf16", 128, 2, False),
                                            ("bf16", 256, 3, True)])
def test_noalloc_forward_equals_forward(prec, l, D, infer):
    K = 2
    big = local_inputs(meshes.sector(6, 16, 10, 4, seed=7), 1, l, K, D, 3)
    small = local_inputs(meshes.sector(4, 12, 6, 4, seed=5), 1, l, K, D, 4)
    assert small["g"]["n_edges"] < big["g"]["n_edges"]
    for name, c in (("larger", big), ("smaller", small)):
        say(f"[noalloc] {prec} l={l} D={D} inference={infer}: {name} graph, {c['g']['n_edges']} edges")
        s = Session(l, K, D, prec, c["g"], c["nf"], c["ef"], c["halo"], c["params"], inference=infer)
        try:
            assert s.ws_bytes <= mgn.MGN_NOALLOC_WS_MAX
            ref = s.forward().cpu().numpy().copy()
            got = _noalloc_out(s)
            assert np.array_equal(got, ref), f"{name}: outputs differ"
            if not infer:
                # the backward of the static-workspace forward equals the one of mgn_forward
                dp_ref = s.backward(c["d_out"])[0].cpu().numpy().copy()
                _noalloc_out(s)
                dp = s.backward(c["d_out"])[0].cpu().numpy()
                assert np.array_equal(dp, dp_ref), f"{name}: gradients differ"
        finally:
            s.close()


def test_noalloc_rejects_oversized_workspace():
    """A graph whose workspace exceeds MGN_NOALLOC_WS_MAX is refused with
    MGN_E_NOMEM and the output is left untouched."""
    c = local_inputs(meshes.sector(20, 16, 40, 4, seed=7), 1, 128, 15, 2, 3)
    s = Session(128, 15, 2, "fp32", c["g"], c["nf"], c["ef"], c["halo"], c["params"])
    try:
        assert s.ws_bytes > mgn.MGN_NOALLOC_WS_MAX
        out = torch.full_like(s.out, 7.0)
        with pytest.raises(mgn.MgnError) as ei:
            mgn.mgn_forward_noalloc(s.model, s.gs, s.node_feat, s.edge_feat, s.halo, out)
        assert ei.value.status == mgn.MGN_E_NOMEM
        torch.cuda.synchronize()
        assert torch.all(out == 7.0)
    finally:
        s.close()

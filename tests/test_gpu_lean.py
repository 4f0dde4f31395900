"""Edge-stream checkpointing (mgn_set_recompute): the backward pass that
recomputes each block's edge latents from the checkpoint below it, its
aggregate by one more edge forward (the last block's is still where the
forward left it, unless a backward has run since), reads the node stream's
bf16 copy and
runs the edge backward (and the edge encoder's) in receiver chunks.  Against
the run that keeps every block's inputs, on the same inputs: outputs bitwise
equal (the forward is the same computation, only stored elsewhere), every
gradient tensor equal up to the order in which chunk sums are added; and
against the oracle with the parity criterion of test_gpu_parity.  And the
first-Linear stash of the row-split kernels (mgn_set_h1_stash): bitwise
the results of the recomputing backward, for every block or only some."""
import numpy as np
import pytest

from synth import meshes
from parity import calibrate, compare, local_inputs, oracle_sensitivity, rel_err, run_gpu, run_oracle, say

pytestmark = pytest.mark.gpu


def _segments_err(shapes, a, b):
    off, worst = 0, (0.0, "")
    for name, _, shape in shapes:
        n = int(np.prod(shape))
        e = rel_err(a[off:off + n], b[off:off + n])
        worst = max(worst, (e, name))
        off += n
    return worst


@pytest.mark.parametrize("l,D", [(64, 3), (128, 2), (256, 3)])
@pytest.mark.parametrize("interval,chunk", [(1, 0), (2, 600), (3, 250)])
def test_checkpointed_equals_stash_all(l, D, interval, chunk):
    K = 5
    say(f"[lean] l={l} D={D} K={K} interval={interval} chunk_edges={chunk}")
    c = local_inputs(meshes.sector(6, 16, 10, 4, seed=7), 1, l, K, D, 3)
    base = run_gpu(c, l, K, D, "bf16")
    lean = run_gpu(c, l, K, D, "bf16", recompute=interval, chunk_edges=chunk)
    assert np.array_equal(base[0], lean[0]), "outputs differ"
    e, name = _segments_err(c["shapes"], lean[1], base[1])
    eh = rel_err(lean[2], base[2])
    say(f"  parameter gradients: worst {e:.2e} ({name}); halo gradient {eh:.2e}")
    assert e <= 1e-4 and eh <= 1e-4


@pytest.mark.parametrize("K,interval", [(5, 2), (4, 4), (1, 1)])
def test_checkpointed_backward_twice(K, interval):
    # the first backward reads the last block's aggregate the forward left;
    # its recompute chains overwrite that slot, so a second backward after
    # the same forward must run that block's edge forward again: both give
    # the same bits, and those of the plan that keeps every block
    from paper_2307_13592_amd.runner import Session
    l, D = 128, 2
    say(f"[lean] backward twice l={l} D={D} K={K} interval={interval}")
    c = local_inputs(meshes.sector(6, 16, 10, 4, seed=13), 1, l, K, D, 6)
    base = run_gpu(c, l, K, D, "bf16")
    s = Session(l, K, D, "bf16", c["g"], c["nf"], c["ef"], c["halo"], c["params"], recompute=interval,
                chunk_edges=300)
    try:
        out = s.forward().cpu().numpy().copy()
        runs = []
        for _ in range(2):
            dp, dh = s.backward(c["d_out"])
            runs.append((dp.cpu().numpy().copy(), dh.cpu().numpy().copy()))
    finally:
        s.close()
    assert np.array_equal(out, base[0]), "outputs differ"
    for name, i in (("parameter gradients", 0), ("halo gradients", 1)):
        assert np.array_equal(runs[0][i], runs[1][i]), f"second backward: {name} differ"
    e, name = _segments_err(c["shapes"], runs[0][0], base[1])
    assert e <= 1e-4 and rel_err(runs[0][1], base[2]) <= 1e-4, (e, name)


def test_checkpointed_against_oracle():
    l, K, D = 128, 4, 2
    say(f"[lean] oracle parity l={l} K={K} D={D}")
    c = local_inputs(meshes.sector(6, 16, 10, 4, seed=11), 1, l, K, D, 5)
    gpu = run_gpu(c, l, K, D, "bf16", recompute=3, chunk_edges=300)
    ref = run_oracle(c, l, K, D, bf16=True)
    bad = compare("checkpointed", "bf16", c["shapes"], gpu, ref, calibrate(c, l, K, D, "bf16"),
                  sens=oracle_sensitivity(c, l, K, D, "bf16"))
    assert not bad, bad


@pytest.mark.parametrize("l,D", [(64, 3), (128, 2)])
@pytest.mark.parametrize("stash", [1, 3, 9])
def test_h1_stash_equals_recompute(l, D, stash):
    K = 3
    say(f"[h1 stash] l={l} D={D} K={K} stash={stash}")
    c = local_inputs(meshes.sector(6, 16, 10, 4, seed=5), 1, l, K, D, 4)
    base = run_gpu(c, l, K, D, "bf16")
    st = run_gpu(c, l, K, D, "bf16", h1_stash=stash)
    for name, a, b in zip(("outputs", "parameter gradients", "halo gradients"), st, base):
        assert np.array_equal(a, b), f"{name} differ: {rel_err(a, b):.2e}"


def test_h1_stash_against_oracle():
    # the inputs of test_checkpointed_against_oracle
    l, K, D = 128, 4, 2
    say(f"[h1 stash] oracle parity l={l} K={K} D={D}")
    c = local_inputs(meshes.sector(6, 16, 10, 4, seed=11), 1, l, K, D, 5)
    gpu = run_gpu(c, l, K, D, "bf16", h1_stash=2)
    ref = run_oracle(c, l, K, D, bf16=True)
    bad = compare("h1 stash", "bf16", c["shapes"], gpu, ref, calibrate(c, l, K, D, "bf16"),
                  sens=oracle_sensitivity(c, l, K, D, "bf16"))
    assert not bad, bad

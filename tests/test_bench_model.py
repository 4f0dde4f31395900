"""The benchmark's accounting (CPU): the algorithmic byte and flop models the
roofline line divides by, written out here from the buffers each kernel
reads and writes, and the rule that a committed traffic summary is used only
for the kernels and stash count it was taken with."""
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import synth  # noqa: E402

E, NO, NH = 27_808_160, 2_000_000, 100_000  # the C4 partition
NL = NO + NH


def test_edge_backward_bytes_c4():
    cfg = synth.CONFIGS["C4"]
    l = cfg.latent
    # stashed launch: reads h_1, de^{k+1} (bf16 rows), receiver and sender
    # ids; writes de^k, dy and dz_0 (bf16 rows); reads dagg and writes the
    # receiver sums of dz_0 once per owned node (fp32 rows)
    stashed = E * (2 * l + 2 * l + 8 + 3 * 2 * l) + NO * 4 * l * 2
    by, fl = bench.algorithmic("edge_bwd", cfg, E, NO, NH, stash=1.0)
    assert by == stashed
    # recomputing launch: reads e^k instead of h_1 and the node projections
    # P (fp32, 2l per local node), and writes h_1 as well
    recomputing = E * (2 * l + 2 * l + 8 + 2 * l + 3 * 2 * l) + NO * 4 * l * 2 + NL * 2 * l * 4
    assert bench.algorithmic("edge_bwd", cfg, E, NO, NH, stash=0.0)[0] == recomputing
    # products: the stashed launch recomputes the last layer and takes the
    # data gradients of both layers and of W_e (3 of the 4 l x l products)
    assert fl == E * 3 * 2 * l * l


def test_edge_forward_and_input_gradient_bytes_c4():
    cfg = synth.CONFIGS["C4"]
    l = cfg.latent
    # forward: reads e^k and the ids per edge, P once per local node; writes
    # e^{k+1} and (stashed blocks) h_1 per edge, agg per owned node
    by, fl = bench.algorithmic("edge_fwd", cfg, E, NO, NH, stash=1.0)
    assert by == E * (2 * l + 8 + 2 * l + 2 * l) + NL * 2 * l * 4 + NO * l * 4
    assert fl == E * 2 * 2 * l * l
    # input gradient: dz_0 rows and transposed-CSR ids per edge, the CSR
    # offsets per local node, dzr, dv read and dv written per owned node,
    # dL/dhalo per halo node, the sender sums written per local node
    by, _ = bench.algorithmic("input_grad", cfg, E, NO, NH)
    assert by == E * (2 * l + 4) + NL * 4 + NO * 4 * l * 3 + NH * 4 * l + NL * 4 * l


def test_step_roofline_fraction():
    cfg = synth.CONFIGS["C4"]
    r = bench.step_roofline(cfg, E, NO, 400.0)
    assert r["bound"] == "hbm"
    assert r["frac"] == pytest.approx(r["roof_ms"] / 400.0)
    # at the roof the fraction is one
    assert bench.step_roofline(cfg, E, NO, r["roof_ms"])["frac"] == pytest.approx(1.0)


def test_traffic_summary_used_only_for_its_kernels(tmp_path, monkeypatch):
    import hashlib
    src = open(os.path.join(ROOT, "paper_2307_13592_amd", "csrc", "kernels.hip"), "rb").read()
    sha = hashlib.sha256(src).hexdigest()
    prof = tmp_path / "profiles"
    prof.mkdir()
    (tmp_path / "paper_2307_13592_amd" / "csrc").mkdir(parents=True)
    (tmp_path / "paper_2307_13592_amd" / "csrc" / "kernels.hip").write_bytes(src)
    body = "h1_stash_blocks: 14\nhbm_bytes_per_launch: 1.5e10\nkernels_sha256: {}\n"
    (prof / "edge_bwd_C4_traffic.txt").write_text(body.format(sha))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.measured_traffic("edge_bwd", "C4", 14) == 1.5e10
    assert bench.measured_traffic("edge_bwd", "C4", 13) is None  # another stash count
    (prof / "edge_bwd_C4_traffic.txt").write_text(body.format("0" * 64))
    assert bench.measured_traffic("edge_bwd", "C4", 14) is None  # other kernels
    assert bench.measured_traffic("edge_fwd", "C4", 14) is None  # no summary

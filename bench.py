"""Benchmark: one MeshGraphNets training step (forward, loss gradient,
backward) on one GPU's mesh partition, through libmgn's C ABI.

Default workload: the 2M-owned-node theta slab of the 100x160x500 swept
sector mesh (100k halo nodes, 27,808,160 local edges), latent 128, 15
message-passing blocks, 2-layer MLPs, bf16 matrix products.  Inputs are
synthetic and seeded, resident in HBM before the timed region.

metric: edge-block updates per second, E * K / step time.  Prints one JSON
line with the roofline position of the dominant kernel and the oracle's
throughput on a bounded sample of the same workload (its CPU baseline).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK = {"hbm": 8.0e12, "bf16": 2.5e15, "fp32": 157.3e12}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def algorithmic(timer: str, cfg, E: int, No: int, Nh: int, lean: bool = False, stash: float = 0.0):
    """Compulsory work of one launch of the kernel class `timer` for one
    block, as (HBM bytes, flops), for the bf16 row-split path the benchmark
    workload takes (latent 64/128, depth 2): each operand row counted once,
    gathered node rows once per node; flops are the MLP products (2 per
    multiply-add).  E edges, No owned and Nh halo nodes; lean: the
    checkpointed plan (the streaming edge backward then recomputes the first
    Linear instead of reading the forward's ReLU output); stash: the share of
    blocks whose row-split forward keeps h_1 for the backward (which then
    reads it in place of e^k and skips the projections, W_e e and the h_1
    write), averaged over the blocks' launches."""
    l, D = cfg.latent, cfg.depth
    Nl = No + Nh
    if cfg.precision != "bf16" or D != 2 or l not in (64, 128):
        # streaming edge kernels (fp32, or l = 256 / depth 3): the concat
        # [e | v_s | v_r] times W_1 per edge; ts bytes per stored element,
        # node rows gathered from the fp32 latents or their bf16 copy
        ts = 2 if cfg.precision == "bf16" else 4
        if timer == "edge_fwd":
            # read e^k, ids, node rows; write e^{k+1}, h_1 (kept for the
            # backward unless lean) and agg
            by = E * ((2 if lean else 3) * ts * l + 8) + Nl * ts * l + No * 4 * l
            return by, E * 2 * l * l * (D + 2)
        if timer == "edge_bwd" and lean:
            # recompute the forward, then the data gradients of every layer
            # and de^k = de^{k+1} + dz_0 W_e: read e^k, de^{k+1} (storage
            # type), ids, node rows, dagg; write de^k, D output gradients and
            # D-1 hidden activations, receiver sums of dz_0
            by = E * (ts * l + ts * l + 8 + ts * l + (2 * D - 1) * ts * l) + Nl * ts * l + No * 4 * l * 2
            return by, E * 4 * l * l * (D + 1)
        if timer == "edge_bwd":
            # from the forward's first-Linear ReLU output h_1: recompute the
            # later layers, then their data gradients and de^k = de^{k+1} +
            # dz_0 W_e: read h_1, de^{k+1} (storage type), ids, dagg; write
            # de^k, D output gradients and D-2 hidden activations, receiver sums
            by = E * (ts * l + ts * l + 8 + ts * l + (2 * D - 2) * ts * l) + No * 4 * l * 2
            return by, E * 2 * l * l * (2 * D - 1)
        return None
    if timer == "edge_bwd":
        # read e^k, de^{k+1} (bf16), receiver / sender ids, dagg rows (fp32),
        # node projections; write de^k, dy, dz_0, h_1 (bf16) and the
        # receiver sums of dz_0; with the stash: read h_1 instead of e^k,
        # no projections, no h_1 write, no W_e e
        by = E * (2 * l + 2 * l + 8 + 2 * l + 3 * 2 * l) + No * l * 4 * 2 + Nl * 2 * l * 4
        by -= stash * (E * 2 * l + Nl * 2 * l * 4)
        return by, E * (4 - stash) * 2 * l * l
    if timer == "edge_fwd":
        # read e^k, ids, projections; write e^{k+1} and agg (and h_1 with the stash)
        by = E * (2 * l + 8 + 2 * l) + Nl * 2 * l * 4 + No * l * 4 + stash * E * 2 * l
        return by, E * 2 * 2 * l * l
    if timer == "node_proj":
        return Nl * (2 * l + 2 * l * 4), Nl * 2 * l * 2 * l
    if timer == "input_grad":
        # dz_0 rows through the transposed CSR, receiver sums, dv (read and
        # write), halo gradients, sender sums out
        by = E * (2 * l + 4) + Nl * 4 + No * l * 4 * 3 + Nh * l * 4 + Nl * l * 4
        return by, Nl * 2 * l * 2 * l
    return None


def step_roofline(cfg, E: int, No: int, ms: float) -> dict:
    """Position of the whole step against the work the method needs per
    edge-block, for kernels that fuse gather, MLP and scatter: flops per
    edge-block forward 2l^2(D+2) + 2l^2(D+1) No/E, forward + backward with
    recompute 4x that; HBM bytes per edge-block forward 2 l s_e + 4, backward
    l s_e + 4 l s_g + 8 (s_e: bytes of a stored edge latent, s_g: of a
    stored edge gradient, both 2 in bf16, 4 in fp32), plus per node and
    block 40 l bytes (forward: v read, agg
    written, v and agg read by the node MLP, v written; backward: v, agg
    and dv read, dv and dagg written), spread over E/No edges.  Roof time =
    the larger of flops / matrix peak and bytes / HBM peak."""
    l, D, K = cfg.latent, cfg.depth, cfg.K
    se = 2 if cfg.precision == "bf16" else 4
    fl = 4 * (2 * l * l * (D + 2) + 2 * l * l * (D + 1) * No / E)
    by = (2 * l * se + 4) + (l * se + 4 * l * se + 8) + 40 * l * No / E
    peak_flops = PEAK["bf16"] if cfg.precision == "bf16" else PEAK["fp32"]
    t_fl, t_by = fl * E * K / peak_flops, by * E * K / PEAK["hbm"]
    roof_s = max(t_fl, t_by)
    return dict(bound="mfma" if t_fl >= t_by else "hbm", flops_per_edge_block=fl, bytes_per_edge_block=by,
                roof_ms=roof_s * 1e3, roof_edges_per_s=E * K / roof_s, frac=roof_s / (ms * 1e-3))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="C4")
    ap.add_argument("--recompute", type=int, default=None,
                    help="edge-stream checkpoint interval (default for C5, whose stash-all workspace exceeds the "
                         "GPU's memory: -1, the smallest interval that fits; 0 otherwise)")
    ap.add_argument("--lockstep", type=int, default=0,
                    help="step P theta slabs of the configuration's whole mesh in lockstep on the one GPU "
                         "(halo exchange after every block), instead of the configuration's single partition")
    ap.add_argument("--inference", action="store_true",
                    help="forward-only rollout steps on the configuration's whole mesh (no halo) instead of the "
                         "training step on its partition")
    ap.add_argument("--nocomm", action="store_true",
                    help="with --lockstep: the paper's NoComm variant (edges across parts dropped, no exchange)")
    ap.add_argument("--precision", default=None, help="override the configuration's precision (fp32 / bf16)")
    ap.add_argument("--graph", action="store_true",
                    help="capture the step into a HIP graph once and time its replays (per-kernel timing and "
                         "the roofline are then omitted: events cannot be read per launch inside a graph)")
    ap.add_argument("--peaks", action="store_true",
                    help="measure what plain streaming kernels and library GEMMs reach on this GPU (the practical "
                         "ceilings beside the spec peaks) and exit")
    ap.add_argument("--h1-stash", type=int, default=-1,
                    help="row-split path: blocks whose first-Linear ReLU output the forward keeps for the "
                         "backward (-1, the default: as many as the GPU's free memory holds)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--oracle-timing", default=None, metavar="CONFIG",
                    help="time only the CPU oracle on CONFIG (whole graph up to --oracle-sample-edges edges, "
                         "else node 0's receptive field) with the OMP_NUM_THREADS the caller sets, and exit")
    ap.add_argument("--oracle-sample-edges", type=int, default=100000)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="after the timed region, copy 1 GiB once (a plain copy kernel of known size, "
                         "for scaling HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py runs on one GPU only: this build has no multi-GPU path (pass --gpus 1)", file=sys.stderr)
        sys.exit(2)

    if args.oracle_timing:
        return oracle_timing(args.oracle_timing, args.oracle_sample_edges)
    import torch
    import synth
    import paper_2307_13592_amd as mgn
    from paper_2307_13592_amd.runner import Session

    if args.peaks:
        return measure_peaks()
    cfg = synth.CONFIGS[args.config]
    if args.precision:
        cfg = synth.Config(**{**cfg.__dict__, "precision": args.precision})
    if args.lockstep:
        return bench_lockstep(args, cfg)
    if args.inference:
        return bench_inference(args, cfg)
    t0 = time.time()
    case = synth.make_case(cfg, region=True)
    mesh = case.mesh
    part = mesh.part if mesh.part is not None else np.zeros(mesh.n_nodes, np.int32)
    g = mgn.mgn_graph_build(mesh.send, mesh.recv, part, mesh.n_nodes, cfg.part)
    loc = case.local_inputs(g["l2g"], g["eperm"], g["n_owned"], g["n_halo"])
    no, nh, ne = g["n_owned"], g["n_halo"], g["n_edges"]
    log(f"[bench] {cfg.name}: {cfg.note}; owned {no}, halo {nh}, edges {ne}; inputs {time.time() - t0:.1f}s")
    recompute = args.recompute if args.recompute is not None else (-1 if cfg.name == "C5" else 0)
    rs = cfg.precision == "bf16" and (cfg.latent == 64 or (cfg.latent == 128 and cfg.depth == 2))
    h1 = args.h1_stash if (rs and recompute == 0) else 0
    sess = Session(cfg.latent, cfg.K, cfg.depth, cfg.precision, g, loc["node_feat"], loc["edge_feat"],
                   loc["halo"], case.params, recompute=recompute, h1_stash=h1)
    recompute = sess.recompute
    stash = min(sess.h1_stash, cfg.K) / cfg.K if (rs and recompute == 0 and cfg.K) else 0.0
    target = torch.as_tensor(loc["target"]).cuda()
    log(f"[bench] workspace {sess.ws_bytes / 2**30:.1f} GiB"
        + (f" (first-Linear stash for {round(stash * cfg.K)} of {cfg.K} blocks)" if stash else "")
        + (f" (checkpoint interval {recompute})" if recompute else ""))

    def step():
        sess.forward()
        _, d_out = sess.mse(target)
        sess.backward(d_out)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log("[bench] warm-up done")
    if args.graph:
        return bench_graph(args, cfg, sess, step, ne, no, nh)
    # timed region: launch timing off, one event pair per step on the launch
    # stream; the step time is the median over the K steps
    stream = torch.cuda.current_stream()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    evs[0].record(stream)
    for i in range(args.steps):
        step()
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    per_step = [evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)]
    ms = float(np.median(per_step))
    ms_mean = evs[0].elapsed_time(evs[-1]) / args.steps
    log(f"[bench] {ms:.2f} ms/step (median of {args.steps}; mean {ms_mean:.2f}, min {min(per_step):.2f}, "
        f"max {max(per_step):.2f})")
    # per-kernel pass, after the timed region: HIP events around every launch
    k_steps = max(1, min(args.steps, 5))
    mgn.mgn_timing_enable(sess.model, True)
    for _ in range(k_steps):
        step()
    torch.cuda.synchronize()
    timers = mgn.mgn_timing_read(sess.model)
    mgn.mgn_timing_enable(sess.model, False)
    for k, (t, n) in sorted(timers.items(), key=lambda kv: -kv[1][0]):
        if n:
            log(f"[bench]   {k:14s} {t / k_steps:9.3f} ms/step  {n // k_steps:4d} launches/step  "
                f"{t / n:8.4f} ms/launch")

    # roofline position of every kernel class with an algorithmic model; the
    # dominant one is the headline's
    peak_flops = PEAK["bf16"] if cfg.precision == "bf16" else PEAK["fp32"]
    kroofs = {}
    for k, (t, n) in timers.items():
        alg = algorithmic(k, cfg, ne, no, nh, lean=recompute > 0, stash=stash) if n else None
        if alg is None:
            continue
        # a block's edge backward may run as several receiver chunks
        # (checkpointed plan): one launch then does its share of the block
        share = cfg.K * k_steps / n if k == "edge_bwd" else 1.0
        by, fl = alg[0] * share, alg[1] * share
        t_launch = t / n * 1e-3
        if fl / by >= peak_flops / PEAK["hbm"]:
            r = dict(bound="mfma", achieved=fl / t_launch / 1e12, peak=peak_flops / 1e12, unit="TFLOP/s")
        else:
            r = dict(bound="hbm", achieved=by / t_launch / 1e9, peak=PEAK["hbm"] / 1e9, unit="GB/s")
        r["frac"] = r["achieved"] / r["peak"]
        r["ms_per_launch"] = t / n
        kroofs[k] = r
    dom = max((k for k in timers if timers[k][1]), key=lambda k: timers[k][0])
    roof = None
    if dom in kroofs:
        roof = {k: v for k, v in kroofs[dom].items() if k != "ms_per_launch"}
        roof["kernel"] = dom
        roof["traffic"] = measured_traffic(dom, cfg.name, round(stash * cfg.K))
    else:
        log(f"[bench] no algorithmic model for {dom} on this configuration: roofline omitted")
    for k, r in sorted(kroofs.items(), key=lambda kv: -timers[kv[0]][0]):
        log(f"[bench]   roofline {k:12s} {r['achieved']:9.1f} {r['unit']:8s} {r['frac']:.3f} of {r['bound']}")
    step_roof = step_roofline(cfg, ne, no, ms)
    log(f"[bench] step at {step_roof['frac']:.3f} of its roof ({step_roof['bound']}-bound, "
        f"{step_roof['roof_ms']:.1f} ms at the peak)")
    if args.copy_calibration:
        src = torch.ones(2 ** 28, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    value = ne * cfg.K / (ms * 1e-3)

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(cfg, g, loc, case)
    sess.close()
    line = {
        "metric": "edges/sec per message-passing step (fwd+bwd)",
        "value": value, "unit": "edge-block updates/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": cfg.precision, "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {cfg.note}", "owned_nodes": no, "halo_nodes": nh, "edges": ne,
                   "latent": cfg.latent, "blocks": cfg.K, "mlp_depth": cfg.depth, "parallelism": "none"},
        "nodes_per_sec": no * cfg.K / (ms * 1e-3),
        "ms_per_step_mean": ms_mean,
        "plan": {"checkpoint_interval": recompute, "h1_stash_blocks": round(stash * cfg.K),
                 "stored": ("every block's edge latents and node stream; the first-Linear ReLU output of "
                            f"{round(stash * cfg.K)} blocks, recomputed from node projections for the other "
                            f"{cfg.K - round(stash * cfg.K)}") if recompute == 0 else
                           (f"edge latents at every {recompute}th block; the others recomputed in the backward")},
        "roofline": roof,
        "kernel_roofline": {k: {kk: vv for kk, vv in v.items()} for k, v in kroofs.items()},
        "step_roofline": step_roof,
        "cpu_baseline": cpu,
        "kernel_ms_per_step": {k: t / k_steps for k, (t, n) in timers.items() if n},
    }
    print(json.dumps(line), flush=True)


def measure_peaks():
    """Practical ceilings: HBM rates of plain streaming kernels (4 GiB
    operands) and the matrix rates of library GEMMs (hipBLASLt through
    torch.matmul, 8192^3), beside the spec peaks."""
    import torch

    def timed(f, n=10):
        f()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(n):
            f()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / n * 1e-3

    N = 2 ** 30  # 4 GiB of fp32
    x = torch.ones(N, device="cuda")
    y = torch.empty_like(x)
    res = {"copy_tb_s": 8 * N / timed(lambda: y.copy_(x)) / 1e12,
           "read_sum_tb_s": 4 * N / timed(lambda: x.sum()) / 1e12,
           "write_fill_tb_s": 4 * N / timed(lambda: y.fill_(1.0)) / 1e12}
    h = N // 2
    z = torch.empty(h, device="cuda")
    res["add_2r1w_tb_s"] = 12 * h / timed(lambda: torch.add(x[:h], x[h:], out=z)) / 1e12
    del x, y, z
    for dt, name in ((torch.bfloat16, "bf16"), (torch.float32, "fp32")):
        n = 8192
        a = torch.randn(n, n, device="cuda").to(dt)
        b = torch.randn(n, n, device="cuda").to(dt)
        res[f"gemm_{name}_tflop_s"] = 2 * n ** 3 / timed(lambda: torch.matmul(a, b), 20) / 1e12
        del a, b
    torch.cuda.empty_cache()
    res["spec"] = {"hbm_tb_s": PEAK["hbm"] / 1e12, "bf16_tflop_s": PEAK["bf16"] / 1e12,
                   "fp32_tflop_s": PEAK["fp32"] / 1e12}
    for k, v in res.items():
        log(f"[bench] {k}: {v}")
    print(json.dumps({"peaks": res}), flush=True)


def bench_graph(args, cfg, sess, step, ne, no, nh):
    """Times replays of the training step captured into one HIP graph."""
    import torch
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    g.replay()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for _ in range(args.steps):
        g.replay()
    ev1.record(stream)
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / args.steps
    log(f"[bench] {ms:.3f} ms/step (HIP graph replays)")
    del g
    sess.close()
    line = {
        "metric": "edges/sec per message-passing step (fwd+bwd)",
        "value": ne * cfg.K / (ms * 1e-3), "unit": "edge-block updates/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": cfg.precision, "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {cfg.note}, step replayed from a HIP graph", "owned_nodes": no,
                   "halo_nodes": nh, "edges": ne, "latent": cfg.latent, "blocks": cfg.K, "mlp_depth": cfg.depth,
                   "parallelism": "none"},
        "nodes_per_sec": no * cfg.K / (ms * 1e-3), "roofline": None, "cpu_baseline": None,
    }
    print(json.dumps(line), flush=True)


def bench_inference(args, cfg):
    """Next-step rollout on the configuration's whole mesh in the forward-only
    plan: one step = forward pass + feeding the prediction back into the
    node features' flow columns."""
    import torch
    import synth
    import paper_2307_13592_amd as mgn
    from paper_2307_13592_amd.runner import Session

    t0 = time.time()
    log(f"[bench] inference: building the whole {cfg.name} mesh ({cfg.note.split(',')[0]})")
    case = synth.make_case(cfg, region=False)
    mesh = case.mesh
    part = np.zeros(mesh.n_nodes, np.int32)
    g = mgn.mgn_graph_build(mesh.send, mesh.recv, part, mesh.n_nodes, 0)
    loc = case.local_inputs(g["l2g"], g["eperm"], g["n_owned"], g["n_halo"])
    no, ne = g["n_owned"], g["n_edges"]
    log(f"[bench] {no} nodes, {ne} edges; inputs {time.time() - t0:.1f}s")
    sess = Session(cfg.latent, cfg.K, cfg.depth, cfg.precision, g, loc["node_feat"], loc["edge_feat"], None,
                   case.params, inference=True)
    log(f"[bench] workspace {sess.ws_bytes / 2**30:.1f} GiB (forward-only plan)")

    def step():
        sess.forward()
        mgn.mgn_rollout_update(sess.out, sess.node_feat)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log("[bench] warm-up done")
    mgn.mgn_timing_enable(sess.model, True)
    stream = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for _ in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / args.steps
    timers = mgn.mgn_timing_read(sess.model)
    sess.close()
    log(f"[bench] {ms:.2f} ms/step")
    for k, (t, n) in sorted(timers.items(), key=lambda kv: -kv[1][0]):
        if n:
            log(f"[bench]   {k:14s} {t / args.steps:9.3f} ms/step  {n // args.steps:4d} launches/step  "
                f"{t / n:8.4f} ms/launch")
    dom = max((k for k in timers if timers[k][1]), key=lambda k: timers[k][0])
    alg = algorithmic(dom, cfg, ne, no, 0)
    roof = None
    if alg is not None:
        t_launch = timers[dom][0] / timers[dom][1] * 1e-3
        roof = dict(bound="hbm", achieved=alg[0] / t_launch / 1e9, peak=PEAK["hbm"] / 1e9, unit="GB/s")
        roof["frac"] = roof["achieved"] / roof["peak"]
        roof["kernel"] = dom
        roof["traffic"] = None
    line = {
        "metric": "edges/sec per message-passing step (forward only)",
        "value": ne * cfg.K / (ms * 1e-3), "unit": "edge-block updates/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": cfg.precision, "data": "synthetic",
        "config": {"workload": f"{cfg.name} whole mesh, next-step rollout (forward-only plan)", "owned_nodes": no,
                   "halo_nodes": 0, "edges": ne, "latent": cfg.latent, "blocks": cfg.K, "mlp_depth": cfg.depth,
                   "parallelism": "none"},
        "nodes_per_sec": no * cfg.K / (ms * 1e-3), "roofline": roof, "cpu_baseline": None,
        "kernel_ms_per_step": {k: t / args.steps for k, (t, n) in timers.items() if n},
    }
    print(json.dumps(line), flush=True)


def bench_lockstep(args, cfg):
    """P theta slabs of the configuration's whole mesh stepped in lockstep on
    one GPU: per block, every part's halo rows are copied from their owners
    (forward) and the halo gradients added back into the owners (backward).
    Loss: the global mean over all parts' owned nodes.  Reports the summed
    throughput and the exchange's share."""
    import torch
    import synth
    import paper_2307_13592_amd as mgn
    from paper_2307_13592_amd.lockstep import Lockstep

    P = args.lockstep
    t0 = time.time()
    log(f"[bench] lockstep: building the whole {cfg.name} mesh ({cfg.note.split(',')[0]})")
    case = synth.make_case(cfg, region=False)
    mesh = case.mesh
    part = mgn.mgn_partition_slabs(mesh.key, P)
    send, recv = mesh.send, mesh.recv
    keep = None
    if args.nocomm:
        keep = np.flatnonzero(part[send] == part[recv])
        send, recv = send[keep], recv[keep]
    graphs = [mgn.mgn_graph_build(send, recv, part, mesh.n_nodes, p) for p in range(P)]
    if keep is not None:  # local edge order -> the mesh's global edge ids
        for g in graphs:
            g["eperm"] = keep[g["eperm"]].astype(np.int32)
    locs = [case.local_inputs(g["l2g"], g["eperm"], g["n_owned"], g["n_halo"]) for g in graphs]
    log(f"[bench] {P} parts: " + ", ".join(f"{g['n_owned']}/{g['n_halo']}/{g['n_edges']}" for g in graphs)
        + f" (owned/halo/edges); inputs {time.time() - t0:.1f}s")
    recompute = args.recompute if args.recompute is not None else (5 if cfg.precision == "bf16" else 0)
    ls = Lockstep(cfg.latent, cfg.K, cfg.depth, cfg.precision, part, graphs, [l["node_feat"] for l in locs],
                  [l["edge_feat"] for l in locs], case.params, recompute=recompute)
    log(f"[bench] workspace {sum(s.ws_bytes for s in ls.sessions) / 2**30:.1f} GiB over {P} parts, "
        f"checkpoint interval {recompute}; {len(ls.links)} exchange links")
    targets = [torch.as_tensor(l["target"]).cuda() for l in locs]

    def step():
        ls.forward()
        _, d_outs = ls.mse(targets)  # the global mean over all parts' owned nodes
        ls.backward(d_outs)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log("[bench] warm-up done")
    for s in ls.sessions:
        mgn.mgn_timing_enable(s.model, True)
    stream = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for _ in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / args.steps
    timers = {}
    for s in ls.sessions:
        for k, (t, n) in mgn.mgn_timing_read(s.model).items():
            a, b = timers.get(k, (0.0, 0))
            timers[k] = (a + t, b + n)
        mgn.mgn_timing_enable(s.model, False)
    ls.close()
    log(f"[bench] {ms:.2f} ms/step")
    for k, (t, n) in sorted(timers.items(), key=lambda kv: -kv[1][0]):
        if n:
            log(f"[bench]   {k:14s} {t / args.steps:9.3f} ms/step  {n // args.steps:5d} launches/step  "
                f"{t / n:8.4f} ms/launch")
    ne = sum(g["n_edges"] for g in graphs)
    no = sum(g["n_owned"] for g in graphs)
    nh = sum(g["n_halo"] for g in graphs)
    ex_ms = timers["exchange"][0] / args.steps
    line = {
        "metric": "edges/sec per message-passing step (fwd+bwd)",
        "value": ne * cfg.K / (ms * 1e-3), "unit": "edge-block updates/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": cfg.precision, "data": "synthetic",
        "config": {"workload": f"{cfg.name} whole mesh, {P} theta slabs in lockstep"
                               + (" without halo (NoComm)" if args.nocomm else ""), "parts": P,
                   "owned_nodes": no, "halo_nodes": nh, "edges": ne, "latent": cfg.latent, "blocks": cfg.K,
                   "mlp_depth": cfg.depth, "checkpoint_interval": recompute, "parallelism": "none"},
        "nodes_per_sec": no * cfg.K / (ms * 1e-3),
        "exchange_ms_per_step": ex_ms, "exchange_share": ex_ms / ms,
        "roofline": None, "cpu_baseline": None,
        "kernel_ms_per_step": {k: t / args.steps for k, (t, n) in timers.items() if n},
    }
    print(json.dumps(line), flush=True)


def measured_traffic(kernel: str, config: str, h1_stash: int = 0):
    """HBM bytes per launch of `kernel` from a committed counter summary
    (profiles/<kernel>_<config>_traffic.txt: FETCH_SIZE and WRITE_SIZE per
    launch, scaled by the counters of a plain copy of known size, averaged
    over the step's launches), used only while the kernels and the number of
    first-Linear stash blocks are the ones the counters were taken with."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"{kernel}_{config}_traffic.txt")
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            vals[k.strip()] = v.strip()
    src = open(os.path.join(ROOT, "paper_2307_13592_amd", "csrc", "kernels.hip"), "rb").read()
    if vals.get("kernels_sha256") != hashlib.sha256(src).hexdigest():
        return None
    if int(vals.get("h1_stash_blocks", "0")) != h1_stash:
        return None
    try:
        return float(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def prefix_sample(g: dict, n_edges: int) -> dict:
    """The first receivers' in-edges, up to about n_edges: receivers keep their
    local ids, senders outside them become halo nodes (ids after the
    receivers, in their original order, so each receiver's edges stay sorted
    by sender).  A bounded sample of a graph's edge-block work for timing."""
    row_ptr = np.asarray(g["row_ptr"], np.int64)
    r = int(np.searchsorted(row_ptr, n_edges))
    r = max(1, min(r, g["n_owned"]))
    ne = int(row_ptr[r])
    send = np.asarray(g["send"][:ne], np.int64)
    outside = np.unique(send[send >= r])
    new = send.copy()
    new[send >= r] = r + np.searchsorted(outside, send[send >= r])
    return dict(n_owned=r, n_halo=int(outside.size), n_edges=ne, row_ptr=row_ptr[:r + 1].astype(np.int32),
                send=new.astype(np.int32), owned=np.arange(r), edges=np.arange(ne))


def oracle_timing(name: str, sample_edges: int):
    """The oracle alone (no GPU) on configuration `name`: the whole graph
    when it has at most `sample_edges` edges, else prefix_sample() of it
    (the cost per edge-block is the measured quantity).  Threads:
    OMP_NUM_THREADS as set by the caller (the oracle's OpenMP runtime reads
    it when it loads)."""
    import oracle
    import synth

    cfg = synth.CONFIGS[name]
    case = synth.make_case(cfg, region=True)
    m = case.mesh
    part = m.part if m.part is not None else np.zeros(m.n_nodes, np.int32)
    t = time.time()
    g = oracle.graph_build(m.send, m.recv, part, m.n_nodes, cfg.part)
    t_graph = time.time() - t
    loc = case.local_inputs(g["l2g"], g["eperm"], g["n_owned"], g["n_halo"])
    if g["n_edges"] <= sample_edges:
        c, what = g, "whole graph"
        nf, ef, halo = loc["node_feat"], loc["edge_feat"], loc["halo"] if g["n_halo"] else None
    else:
        c, what = prefix_sample(g, sample_edges), "first receivers' in-edges"
        nf, ef = loc["node_feat"][c["owned"]], loc["edge_feat"][c["edges"]]
        halo = synth.halo_latents(cfg.K, c["n_halo"], cfg.latent, cfg.seed) if c["n_halo"] else None
    d_out = np.random.default_rng([cfg.seed, 5]).standard_normal((c["n_owned"], 5))
    ocfg = oracle.ModelCfg(cfg.latent, cfg.K, cfg.depth, bf16=cfg.precision == "bf16")
    t = time.time()
    oracle.step(ocfg, c, case.params.astype(np.float64), nf.astype(np.float64), ef.astype(np.float64),
                None if halo is None else halo.astype(np.float64), d_out)
    dt = time.time() - t
    threads = os.environ.get("OMP_NUM_THREADS", "unset (all cores)")
    res = {"oracle_timing": {"config": name, "sample": f"{what}: {c['n_owned']} owned + {c['n_halo']} halo nodes, "
                                                      f"{c['n_edges']} edges, {cfg.K} blocks, fwd+bwd",
                             "seconds": dt, "edge_block_updates_per_s": c["n_edges"] * cfg.K / dt,
                             "nodes_per_s": c["n_owned"] * cfg.K / dt, "graph_build_s": t_graph,
                             "omp_num_threads": threads, "cpu_model": cpu_model(),
                             "host_cpus": os.cpu_count()}}
    log(f"[bench] oracle {name}: {res['oracle_timing']['sample']} in {dt:.2f}s ({threads} threads)")
    print(json.dumps(res), flush=True)


def cpu_baseline(cfg, g, loc, case):
    """The oracle on a bounded sample of the workload: the receptive field of
    one corner node (every block's edges into nodes within K-1 hops), which is
    what one output and, with the loss gradient on that node, its share of the
    parameter gradients depend on."""
    import oracle
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    from cone import cone

    c = cone(g, [0], cfg.K)
    ef = loc["edge_feat"][c["edges"]]
    nf = loc["node_feat"][c["owned"]]
    halo = loc["halo"][:, c["halo"]] if c["n_halo"] else None
    d_out = np.zeros((c["n_owned"], 5))
    d_out[c["centers_sub"]] = 1.0
    ocfg = oracle.ModelCfg(cfg.latent, cfg.K, cfg.depth, bf16=cfg.precision == "bf16")
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    t = time.time()
    oracle.step(ocfg, c, case.params.astype(np.float64), nf.astype(np.float64), ef.astype(np.float64),
                None if halo is None else halo.astype(np.float64), d_out)
    dt = time.time() - t
    log(f"[bench] oracle sample: {c['n_edges']} edges x {cfg.K} blocks in {dt:.1f}s ({threads} threads)")
    return {"value": c["n_edges"] * cfg.K / dt, "unit": "edge-block updates/s", "cores": threads,
            "kind": "oracle", "cpu_model": cpu_model(),
            "sample": f"receptive field of one corner node: {c['n_owned']} owned + {c['n_halo']} halo nodes, "
                      f"{c['n_edges']} edges, all {cfg.K} blocks, fwd+bwd"}


if __name__ == "__main__":
    main()

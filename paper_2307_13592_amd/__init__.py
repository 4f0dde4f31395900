"""Python binding of libmgn (include/mgn.h): one MeshGraphNets training step
on one MI355X mesh partition.

The functions here carry the C ABI's names and only marshal arguments
(torch device tensors -> device pointers, numpy arrays -> host pointers,
status codes -> exceptions).  Every step of the computation runs in the HIP
kernels of libmgn.so; there is no fallback.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

from . import build as _build

MGN_OK, MGN_E_ARG, MGN_E_GRAPH, MGN_E_STATE, MGN_E_NOMEM, MGN_E_HIP, MGN_E_UNSUPPORTED = range(7)
MGN_FP32, MGN_BF16 = 0, 1
STATUS_NAMES = ["MGN_OK", "MGN_E_ARG", "MGN_E_GRAPH", "MGN_E_STATE", "MGN_E_NOMEM", "MGN_E_HIP", "MGN_E_UNSUPPORTED"]

# every symbol include/mgn.h declares
EXPORTS = ["mgn_create", "mgn_destroy", "mgn_last_error", "mgn_param_count", "mgn_set_params", "mgn_sgd_step",
           "mgn_get_params",
           "mgn_partition_slabs", "mgn_graph_sizes", "mgn_graph_build", "mgn_graph_validate", "mgn_set_recompute",
           "mgn_set_inference", "mgn_set_h1_stash", "mgn_rollout_update", "mgn_norm_accumulate", "mgn_norm_apply",
           "mgn_workspace_size",
           "mgn_forward", "mgn_backward", "mgn_forward_begin", "mgn_forward_block", "mgn_forward_end",
           "mgn_backward_begin", "mgn_backward_block", "mgn_backward_end", "mgn_halo_masks", "mgn_copy_latents",
           "mgn_add_latent_grads", "mgn_lockstep_forward", "mgn_lockstep_backward", "mgn_mse_grad",
           "mgn_mse_grad_global", "mgn_timing_enable", "mgn_timing_read", "mgn_forward_noalloc"]
TIMERS = ["encode", "edge_fwd", "node_fwd", "decode", "edge_bwd", "node_bwd", "input_grad", "weight_grad",
          "other", "node_proj", "exchange"]


class MgnError(RuntimeError):
    def __init__(self, status: int, msg: str):
        self.status = status
        name = STATUS_NAMES[status] if 0 <= status < len(STATUS_NAMES) else str(status)
        super().__init__(f"{name}: {msg}")


class mgn_config(C.Structure):
    _fields_ = [("latent", C.c_int32), ("n_blocks", C.c_int32), ("depth", C.c_int32), ("node_in", C.c_int32),
                ("edge_in", C.c_int32), ("node_out", C.c_int32), ("precision", C.c_int32), ("ln_eps", C.c_float)]


class mgn_halo_link(C.Structure):
    _fields_ = [("part", C.c_int32), ("owner", C.c_int32), ("recv_idx", C.c_void_p), ("send_rows", C.c_void_p),
                ("n", C.c_int64)]


class mgn_graph(C.Structure):
    _fields_ = [("n_owned", C.c_int64), ("n_halo", C.c_int64), ("n_edges", C.c_int64), ("row_ptr", C.c_void_p),
                ("send", C.c_void_p), ("trow_ptr", C.c_void_p), ("tedge", C.c_void_p)]


_lib = None


def lib() -> C.CDLL:
    """Loads libmgn.so, building it first only if no build exists."""
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        L = C.CDLL(_build.LIB)
        for name in EXPORTS:
            getattr(L, name)
        vp, i64, i32 = C.c_void_p, C.c_int64, C.c_int32
        sig = {
            "mgn_create": (C.c_int, [vp, vp]),
            "mgn_destroy": (None, [vp]),
            "mgn_last_error": (C.c_char_p, [vp]),
            "mgn_param_count": (i64, [vp]),
            "mgn_set_params": (C.c_int, [vp, vp, C.c_int, vp]),
            "mgn_get_params": (C.c_int, [vp, vp, C.c_int, vp]),
            "mgn_sgd_step": (C.c_int, [vp, vp, C.c_float, vp]),
            "mgn_partition_slabs": (C.c_int, [vp, i64, i32, vp]),
            "mgn_graph_sizes": (C.c_int, [vp, vp, i64, vp, i64, i32, vp]),
            "mgn_graph_build": (C.c_int, [vp, vp, i64, vp, i64, i32, vp, vp, vp, vp, vp, vp]),
            "mgn_graph_validate": (C.c_int, [vp, vp, vp]),
            "mgn_set_recompute": (C.c_int, [vp, i32, i64]),
            "mgn_set_inference": (C.c_int, [vp, i32]),
            "mgn_set_h1_stash": (C.c_int, [vp, i32]),
            "mgn_rollout_update": (C.c_int, [vp, i64, i32, vp, i32, i32, vp]),
            "mgn_norm_accumulate": (C.c_int, [vp, i64, i32, vp, vp, vp]),
            "mgn_norm_apply": (C.c_int, [vp, i64, i32, vp, C.c_double, vp, vp]),
            "mgn_workspace_size": (C.c_int, [vp, vp, vp]),
            "mgn_forward": (C.c_int, [vp, vp, vp, vp, vp, vp, vp, C.c_size_t, vp]),
            "mgn_backward": (C.c_int, [vp, vp, vp, C.c_int, vp, vp]),
            "mgn_forward_noalloc": (C.c_int, [vp, vp, vp, vp, vp, vp, vp]),
            "mgn_forward_begin": (C.c_int, [vp, vp, vp, vp, vp, vp, vp, C.c_size_t, vp]),
            "mgn_forward_block": (C.c_int, [vp, vp]),
            "mgn_forward_end": (C.c_int, [vp, vp]),
            "mgn_backward_begin": (C.c_int, [vp, vp, vp, C.c_int, vp, vp]),
            "mgn_backward_block": (C.c_int, [vp, vp]),
            "mgn_backward_end": (C.c_int, [vp, vp]),
            "mgn_halo_masks": (C.c_int, [vp, i64, i64, vp, i64, vp, i64, i32, vp, vp, vp]),
            "mgn_copy_latents": (C.c_int, [vp, vp, vp, i64, vp, i64, vp]),
            "mgn_add_latent_grads": (C.c_int, [vp, vp, i64, vp, vp, i64, vp]),
            "mgn_lockstep_forward": (C.c_int, [i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, i32, vp]),
            "mgn_lockstep_backward": (C.c_int, [i32, vp, vp, vp, C.c_int, vp, vp, i32, vp]),
            "mgn_mse_grad": (C.c_int, [vp, vp, vp, i64, i32, vp, vp, vp]),
            "mgn_mse_grad_global": (C.c_int, [vp, vp, vp, i64, i32, i64, vp, vp, vp]),
            "mgn_timing_enable": (C.c_int, [vp, C.c_int]),
            "mgn_timing_read": (C.c_int, [vp, C.c_int, vp, vp]),
        }
        for name, (res, args) in sig.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


# ------------------------------------------------------------ marshalling ---
def _dev(t):
    """Device pointer of a torch tensor (None -> NULL)."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("expected a device tensor")
    if not t.is_contiguous():
        raise ValueError("expected a contiguous tensor")
    return C.c_void_p(t.data_ptr())


def _devt(t, dtype, name: str, shape=None, numel=None, min_numel=None):
    """_dev with the checks the C ABI cannot make (it takes no dtype, and
    no length for some buffers): torch dtype, exact shape, exact or minimum
    element count."""
    if t is None:
        raise ValueError(f"{name}: expected a device tensor, got None")
    if t.dtype != dtype:
        raise ValueError(f"{name}: expected {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: expected shape {tuple(shape)}, got {tuple(t.shape)}")
    if numel is not None and t.numel() != numel:
        raise ValueError(f"{name}: expected {numel} elements, got {t.numel()}")
    if min_numel is not None and t.numel() < min_numel:
        raise ValueError(f"{name}: expected at least {min_numel} elements, got {t.numel()}")
    return _dev(t)


def _host(a, dtype):
    if a is None:
        return None, None
    a = np.ascontiguousarray(a, dtype=dtype)
    return a, a.ctypes.data_as(C.c_void_p)


def _stream(stream):
    if stream is None:
        import torch
        return C.c_void_p(torch.cuda.current_stream().cuda_stream)
    return C.c_void_p(int(stream))


def _check(st: int, model=None):
    if st != MGN_OK:
        msg = lib().mgn_last_error(model).decode()
        raise MgnError(st, msg)


# ------------------------------------------------------------------- ABI ---
def mgn_create(latent: int, n_blocks: int, depth: int, precision: int = MGN_FP32, node_in: int = 11,
               edge_in: int = 4, node_out: int = 5, ln_eps: float = 1e-5) -> C.c_void_p:
    cfg = mgn_config(latent, n_blocks, depth, node_in, edge_in, node_out, precision, ln_eps)
    h = C.c_void_p()
    _check(lib().mgn_create(C.byref(cfg), C.byref(h)))
    return h


def mgn_destroy(model) -> None:
    lib().mgn_destroy(model)


def mgn_last_error(model=None) -> str:
    return lib().mgn_last_error(model).decode()


def mgn_param_count(model) -> int:
    return int(lib().mgn_param_count(model))


def mgn_set_params(model, params, stream=None) -> None:
    """params: float32 device tensor or host array of mgn_param_count entries."""
    if hasattr(params, "is_cuda") and params.is_cuda:
        _check(lib().mgn_set_params(model, _dev(params), 1, _stream(stream)), model)
    else:
        a, p = _host(params, np.float32)
        if a.size != mgn_param_count(model):
            raise ValueError("parameter vector has the wrong length")
        _check(lib().mgn_set_params(model, p, 0, _stream(stream)), model)


def mgn_sgd_step(model, grad, lr: float, stream=None) -> None:
    """params -= lr * grad on the device (grad: float32 device tensor)."""
    if grad.numel() != mgn_param_count(model):
        raise ValueError("gradient vector has the wrong length")
    _check(lib().mgn_sgd_step(model, _dev(grad), float(lr), _stream(stream)), model)


def mgn_get_params(model, stream=None) -> np.ndarray:
    out = np.empty(mgn_param_count(model), np.float32)
    _check(lib().mgn_get_params(model, out.ctypes.data_as(C.c_void_p), 0, _stream(stream)), model)
    return out


def mgn_partition_slabs(key, nparts: int) -> np.ndarray:
    k, kp = _host(key, np.int32)
    part = np.empty(k.shape[0], np.int32)
    _check(lib().mgn_partition_slabs(kp, k.shape[0], nparts, part.ctypes.data_as(C.c_void_p)))
    return part


def mgn_graph_sizes(send, recv, part, n_nodes: int, p: int):
    s, sp = _host(send, np.int32)
    r, rp = _host(recv, np.int32)
    pa, pp = _host(part, np.int32)
    sz = np.zeros(3, np.int64)
    _check(lib().mgn_graph_sizes(sp, rp, s.shape[0], pp, n_nodes, p, sz.ctypes.data_as(C.c_void_p)))
    return tuple(int(x) for x in sz)


def mgn_graph_build(send, recv, part, n_nodes: int, p: int) -> dict:
    """Host-side build of part p's local graph; returns numpy arrays."""
    no, nh, ne = mgn_graph_sizes(send, recv, part, n_nodes, p)
    s, sp = _host(send, np.int32)
    r, rp = _host(recv, np.int32)
    pa, pp = _host(part, np.int32)
    g = dict(n_owned=no, n_halo=nh, n_edges=ne, row_ptr=np.empty(no + 1, np.int32), send=np.empty(ne, np.int32),
             eperm=np.empty(ne, np.int32), trow_ptr=np.empty(no + nh + 1, np.int32), tedge=np.empty(ne, np.int32),
             l2g=np.empty(no + nh, np.int32))
    ptr = lambda k: g[k].ctypes.data_as(C.c_void_p)
    _check(lib().mgn_graph_build(sp, rp, s.shape[0], pp, n_nodes, p, ptr("row_ptr"), ptr("send"), ptr("eperm"),
                                 ptr("trow_ptr"), ptr("tedge"), ptr("l2g")))
    return g


def graph_struct(dg: dict) -> mgn_graph:
    """mgn_graph from a dict of sizes and int32 device tensors."""
    return mgn_graph(dg["n_owned"], dg["n_halo"], dg["n_edges"], _dev(dg["row_ptr"]), _dev(dg["send"]),
                     _dev(dg["trow_ptr"]), _dev(dg["tedge"]))


def mgn_graph_validate(model, graph: mgn_graph, stream=None) -> None:
    _check(lib().mgn_graph_validate(model, C.byref(graph), _stream(stream)), model)


def mgn_set_recompute(model, interval: int, chunk_edges: int = 0) -> None:
    _check(lib().mgn_set_recompute(model, int(interval), int(chunk_edges)), model)


def mgn_set_inference(model, on: bool = True) -> None:
    _check(lib().mgn_set_inference(model, int(bool(on))), model)


def mgn_set_h1_stash(model, n_blocks: int) -> None:
    _check(lib().mgn_set_h1_stash(model, int(n_blocks)), model)


MGN_NORM_MAX_COLS = 64
MGN_NORM_WORK_PER_COL = 1024


def mgn_norm_accumulate(x, stats, work, stream=None) -> None:
    """Adds the rows of x (device float32 [rows][cols]) to the running
    statistics `stats` (device float64 [1 + 2 cols]); work: device float64
    scratch of at least MGN_NORM_WORK_PER_COL * cols."""
    import torch
    if x.dim() != 2:
        raise ValueError("x: expected [rows][cols]")
    rows, cols = x.shape
    _check(lib().mgn_norm_accumulate(_devt(x, torch.float32, "x"), rows, cols,
                                     _devt(stats, torch.float64, "stats", numel=1 + 2 * cols),
                                     _devt(work, torch.float64, "work", min_numel=MGN_NORM_WORK_PER_COL * cols),
                                     _stream(stream)))


def mgn_norm_apply(x, stats, out, eps: float = 1e-8, stream=None) -> None:
    """out = (x - mean) / max(std, eps) per column (device float32; out may be x)."""
    import torch
    if x.dim() != 2:
        raise ValueError("x: expected [rows][cols]")
    rows, cols = x.shape
    _check(lib().mgn_norm_apply(_devt(x, torch.float32, "x"), rows, cols,
                                _devt(stats, torch.float64, "stats", numel=1 + 2 * cols), C.c_double(eps),
                                _devt(out, torch.float32, "out", shape=(rows, cols)), _stream(stream)))


def mgn_rollout_update(out, node_feat, col0: int = 3, stream=None) -> None:
    """node_feat[:, col0:col0 + out.shape[1]] += out (device tensors)."""
    import torch
    n, d = out.shape
    if node_feat.dim() != 2 or node_feat.shape[0] != n:
        raise ValueError("node_feat: expected [n][features] with the rows of out")
    _check(lib().mgn_rollout_update(_devt(out, torch.float32, "out"), n, d,
                                    _devt(node_feat, torch.float32, "node_feat"), int(node_feat.shape[1]), int(col0),
                                    _stream(stream)))


def mgn_workspace_size(model, graph: mgn_graph) -> int:
    n = C.c_size_t()
    _check(lib().mgn_workspace_size(model, C.byref(graph), C.byref(n)), model)
    return int(n.value)


def mgn_forward(model, graph: mgn_graph, node_feat, edge_feat, halo, out, workspace, stream=None) -> None:
    _check(lib().mgn_forward(model, C.byref(graph), _dev(node_feat), _dev(edge_feat), _dev(halo), _dev(out),
                             _dev(workspace), workspace.numel() * workspace.element_size(), _stream(stream)),
           model)


MGN_NOALLOC_WS_MAX = 128 << 20


def mgn_forward_noalloc(model, graph: mgn_graph, node_feat, edge_feat, halo, out, stream=None) -> None:
    """mgn_forward with the library's static per-GPU workspace (no caller
    workspace, no allocation)."""
    _check(lib().mgn_forward_noalloc(model, C.byref(graph), _dev(node_feat), _dev(edge_feat), _dev(halo), _dev(out),
                                     _stream(stream)), model)


def mgn_backward(model, d_out, d_params, accumulate: bool = False, d_halo=None, stream=None) -> None:
    _check(lib().mgn_backward(model, _dev(d_out), _dev(d_params), int(bool(accumulate)), _dev(d_halo),
                              _stream(stream)), model)


def mgn_forward_begin(model, graph: mgn_graph, node_feat, edge_feat, halo, out, workspace, stream=None) -> None:
    _check(lib().mgn_forward_begin(model, C.byref(graph), _dev(node_feat), _dev(edge_feat), _dev(halo), _dev(out),
                                   _dev(workspace), workspace.numel() * workspace.element_size(), _stream(stream)),
           model)


def mgn_forward_block(model, stream=None) -> None:
    _check(lib().mgn_forward_block(model, _stream(stream)), model)


def mgn_forward_end(model, stream=None) -> None:
    _check(lib().mgn_forward_end(model, _stream(stream)), model)


def mgn_backward_begin(model, d_out, d_params, accumulate: bool = False, d_halo=None, stream=None) -> None:
    _check(lib().mgn_backward_begin(model, _dev(d_out), _dev(d_params), int(bool(accumulate)), _dev(d_halo),
                                    _stream(stream)), model)


def mgn_backward_block(model, stream=None) -> None:
    _check(lib().mgn_backward_block(model, _stream(stream)), model)


def mgn_backward_end(model, stream=None) -> None:
    _check(lib().mgn_backward_end(model, _stream(stream)), model)


def mgn_halo_masks(l2g_p, n_owned_p: int, part, l2g_q, n_owned_q: int, q: int):
    """Host exchange lists of part p's halo nodes owned by part q:
    (recv_idx, send_rows) int32 arrays (halo index in p, local id in q)."""
    lp, lpp = _host(l2g_p, np.int32)
    pa, pp = _host(part, np.int32)
    lq, lqp = _host(l2g_q, np.int32)
    nh = lp.shape[0] - int(n_owned_p)
    recv = np.empty(max(nh, 0), np.int32)
    send = np.empty(max(nh, 0), np.int32)
    cnt = C.c_int64()
    _check(lib().mgn_halo_masks(lpp, int(n_owned_p), nh, pp, pa.shape[0], lqp, int(n_owned_q), int(q),
                                recv.ctypes.data_as(C.c_void_p), send.ctypes.data_as(C.c_void_p), C.byref(cnt)))
    return recv[:cnt.value].copy(), send[:cnt.value].copy()


def mgn_copy_latents(owner, send_rows, recv_idx, halo_k, stream=None) -> None:
    """halo_k[recv_idx[i]] = owner's current node latents[send_rows[i]] (device tensors)."""
    _check(lib().mgn_copy_latents(owner, _dev(send_rows), _dev(recv_idx), int(send_rows.numel()), _dev(halo_k),
                                  int(halo_k.shape[0]), _stream(stream)), owner)


def mgn_add_latent_grads(owner, d_halo_k, recv_idx, send_rows, stream=None) -> None:
    """owner's dL/dv[send_rows[i]] += d_halo_k[recv_idx[i]] (device tensors)."""
    _check(lib().mgn_add_latent_grads(owner, _dev(d_halo_k), int(d_halo_k.shape[0]), _dev(recv_idx),
                                      _dev(send_rows), int(send_rows.numel()), _stream(stream)), owner)


def _ptrs(ts):
    """C array of device pointers (NULL for None)."""
    return (C.c_void_p * len(ts))(*[None if t is None else t.data_ptr() for t in ts])


def mgn_lockstep_forward(models, graphs, node_feats, edge_feats, halos, outs, workspaces, links,
                         stream=None) -> None:
    """models, graphs (mgn_graph), device tensors per part; links: list of
    (part, owner, recv_idx, send_rows) with device int32 index tensors."""
    P = len(models)
    ms = (C.c_void_p * P)(*[m.value for m in models])
    gs = (mgn_graph * P)(*graphs)
    lk = (mgn_halo_link * max(len(links), 1))(*[mgn_halo_link(p, q, r.data_ptr(), s.data_ptr(), r.numel())
                                                 for p, q, r, s in links])
    wb = (C.c_size_t * P)(*[w.numel() * w.element_size() for w in workspaces])
    st = lib().mgn_lockstep_forward(P, ms, gs, _ptrs(node_feats), _ptrs(edge_feats), _ptrs(halos), _ptrs(outs),
                                    _ptrs(workspaces), wb, lk, len(links), _stream(stream))
    _check(st)


def mgn_lockstep_backward(models, d_outs, d_params, d_halos, links, accumulate: bool = False, stream=None) -> None:
    P = len(models)
    ms = (C.c_void_p * P)(*[m.value for m in models])
    lk = (mgn_halo_link * max(len(links), 1))(*[mgn_halo_link(p, q, r.data_ptr(), s.data_ptr(), r.numel())
                                                 for p, q, r, s in links])
    st = lib().mgn_lockstep_backward(P, ms, _ptrs(d_outs), _dev(d_params), int(bool(accumulate)), _ptrs(d_halos),
                                     lk, len(links), _stream(stream))
    _check(st)


def _mse_args(out, target, mask, loss, d_out):
    import torch
    if out.dim() != 2:
        raise ValueError("out: expected [n][d]")
    n, d = out.shape
    return (n, d, _devt(out, torch.float32, "out"), _devt(target, torch.float32, "target", shape=(n, d)),
            None if mask is None else _devt(mask, torch.uint8, "mask", numel=n),
            _devt(loss, torch.float32, "loss", min_numel=2), _devt(d_out, torch.float32, "d_out", shape=(n, d)))


def mgn_mse_grad(out, target, mask, loss, d_out, stream=None) -> None:
    n, d, po, pt, pm, pl, pd = _mse_args(out, target, mask, loss, d_out)
    _check(lib().mgn_mse_grad(po, pt, pm, n, d, pl, pd, _stream(stream)))


def mgn_mse_grad_global(out, target, mask, global_rows: int, loss, d_out, stream=None) -> None:
    n, d, po, pt, pm, pl, pd = _mse_args(out, target, mask, loss, d_out)
    _check(lib().mgn_mse_grad_global(po, pt, pm, n, d, int(global_rows), pl, pd, _stream(stream)))


def mgn_timing_enable(model, enable: bool = True) -> None:
    _check(lib().mgn_timing_enable(model, int(bool(enable))), model)


def mgn_timing_read(model) -> dict:
    """{timer name: (total ms, launches)} for every timer class."""
    res = {}
    for i, name in enumerate(TIMERS):
        ms, n = C.c_double(), C.c_int64()
        _check(lib().mgn_timing_read(model, i, C.byref(ms), C.byref(n)), model)
        res[name] = (ms.value, n.value)
    return res

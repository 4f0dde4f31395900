"""CPU oracle for the MeshGraphNets training step -- TEST INFRASTRUCTURE.

ctypes wrapper around oracle/liboracle.so (built from mgn_oracle.cpp with g++).
Only the tests, the smoke check and the CPU-baseline leg of the benchmark may
import this.  Everything it returns is float64.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass

import numpy as np

from . import build as _build

_lib = None


class orc_cfg(C.Structure):
    _fields_ = [("latent", C.c_int32), ("n_blocks", C.c_int32), ("depth", C.c_int32),
                ("node_in", C.c_int32), ("edge_in", C.c_int32), ("node_out", C.c_int32),
                ("ln_eps", C.c_double), ("bf16", C.c_int32)]


@dataclass
class ModelCfg:
    latent: int
    n_blocks: int
    depth: int
    node_in: int = 11
    edge_in: int = 4
    node_out: int = 5
    ln_eps: float = 1e-5
    bf16: bool = False   # mixed-precision reading: bfloat16 operands of every matrix product

    def c(self) -> orc_cfg:
        return orc_cfg(self.latent, self.n_blocks, self.depth, self.node_in, self.edge_in,
                       self.node_out, self.ln_eps, int(self.bf16))


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        L = C.CDLL(_build.LIB)
        L.orc_param_count.restype = C.c_int64
        _lib = L
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def _f64(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.float64)


def param_count(cfg: ModelCfg) -> int:
    c = cfg.c()
    return int(lib().orc_param_count(C.byref(c)))


def partition(key, nparts: int) -> np.ndarray:
    key = _i32(key)
    part = np.empty(key.shape[0], np.int32)
    rc = lib().orc_partition(_p(key), C.c_int64(key.shape[0]), C.c_int32(nparts), _p(part))
    if rc:
        raise ValueError("orc_partition rejected its arguments")
    return part


def graph_build(send, recv, part, n_nodes: int, p: int) -> dict:
    send, recv, part = _i32(send), _i32(recv), _i32(part)
    sz = np.zeros(3, np.int64)
    ne_g = C.c_int64(send.shape[0])
    rc = lib().orc_graph_sizes(_p(send), _p(recv), ne_g, _p(part), C.c_int64(n_nodes), C.c_int32(p), _p(sz))
    if rc:
        raise ValueError("orc_graph_sizes rejected its arguments")
    no, nh, ne = (int(x) for x in sz)
    g = dict(n_owned=no, n_halo=nh, n_edges=ne,
             row_ptr=np.empty(no + 1, np.int32), send=np.empty(ne, np.int32), eperm=np.empty(ne, np.int32),
             trow_ptr=np.empty(no + nh + 1, np.int32), tedge=np.empty(ne, np.int32),
             l2g=np.empty(no + nh, np.int32))
    rc = lib().orc_graph_build(_p(send), _p(recv), ne_g, _p(part), C.c_int64(n_nodes), C.c_int32(p),
                               _p(g["row_ptr"]), _p(g["send"]), _p(g["eperm"]), _p(g["trow_ptr"]),
                               _p(g["tedge"]), _p(g["l2g"]))
    if rc:
        raise ValueError("orc_graph_build rejected its arguments")
    return g


def edge_features(coords, send, recv, h: float) -> np.ndarray:
    coords, send, recv = _f64(coords), _i32(send), _i32(recv)
    out = np.empty((send.shape[0], 4), np.float64)
    if lib().orc_edge_features(_p(coords), _p(send), _p(recv), C.c_int64(send.shape[0]), C.c_double(h), _p(out)):
        raise ValueError("orc_edge_features rejected its arguments")
    return out


def scatter_sum(row_ptr, m) -> np.ndarray:
    row_ptr, m = _i32(row_ptr), _f64(m)
    n = row_ptr.shape[0] - 1
    out = np.empty((n, m.shape[1]), np.float64)
    if lib().orc_scatter_sum(C.c_int64(n), _p(row_ptr), _p(m), C.c_int32(m.shape[1]), _p(out)):
        raise ValueError("orc_scatter_sum rejected its arguments")
    return out


def step(cfg: ModelCfg, g: dict, params, node_feat, edge_feat, halo=None, d_out=None,
         want_v: bool = False, want_e: bool = False) -> dict:
    """Forward (and backward when d_out is given) on a partition-local graph g
    (keys n_owned, n_halo, n_edges, row_ptr, send)."""
    no, nh, ne = g["n_owned"], g["n_halo"], g["n_edges"]
    l, K = cfg.latent, cfg.n_blocks
    params = _f64(params)
    nf = _f64(np.asarray(node_feat).reshape(no, cfg.node_in))
    ef = _f64(np.asarray(edge_feat).reshape(ne, cfg.edge_in))
    halo = _f64(halo) if (halo is not None and nh > 0) else None
    d_out = _f64(d_out)
    res = dict(out=np.empty((no, cfg.node_out), np.float64))
    if d_out is not None:
        res["d_params"] = np.empty(param_count(cfg), np.float64)
        res["d_halo"] = np.empty((K, nh, l), np.float64)
    if want_v:
        res["v_all"] = np.empty((K + 1, no + nh, l), np.float64)
    if want_e:
        res["e_all"] = np.empty((K + 1, ne, l), np.float64)
    c = cfg.c()
    rc = lib().orc_step(C.byref(c), C.c_int64(no), C.c_int64(nh), C.c_int64(ne),
                        _p(_i32(g["row_ptr"])), _p(_i32(g["send"])), _p(params), _p(nf), _p(ef),
                        _p(halo), _p(d_out), _p(res["out"]), _p(res.get("d_params")),
                        _p(res.get("d_halo")), _p(res.get("v_all")), _p(res.get("e_all")))
    if rc:
        raise ValueError("orc_step rejected its arguments")
    return res


def mse_grad(out, target, mask=None, global_rows: int = 0):
    """Masked mean squared error and its gradient; with global_rows > 0 this
    part's share of the mean over global_rows rows of all parts."""
    out, target = _f64(out), _f64(target)
    n, d = out.shape
    m = None if mask is None else np.ascontiguousarray(mask, dtype=np.uint8)
    loss = np.zeros(1, np.float64)
    dout = np.empty_like(out)
    if lib().orc_mse_grad_global(_p(out), _p(target), _p(m), C.c_int64(n), C.c_int32(d), C.c_int64(global_rows),
                                 _p(loss), _p(dout)):
        raise ValueError("orc_mse_grad_global rejected its arguments")
    return float(loss[0]), dout


def sgd_step(params, grad, lr: float) -> np.ndarray:
    """Algorithm 1's update: params - lr * grad (float64, new array)."""
    out = _f64(params).copy()
    g = _f64(grad)
    if out.shape != g.shape or lib().orc_sgd_step(_p(out), _p(g), C.c_int64(out.size), C.c_double(lr)):
        raise ValueError("orc_sgd_step rejected its arguments")
    return out


def rollout_update(node_feat, out, col0: int = 3) -> np.ndarray:
    """Next-step input: the flow columns of node_feat plus the predicted
    increment out (float64, new array)."""
    nf = _f64(node_feat).copy()
    o = _f64(out)
    n, fin = nf.shape
    if o.shape[0] != n or lib().orc_rollout_update(_p(nf), C.c_int64(n), C.c_int32(fin), _p(o),
                                                   C.c_int32(o.shape[1]), C.c_int32(col0)):
        raise ValueError("orc_rollout_update rejected its arguments")
    return nf


def norm_accumulate(stats, x) -> np.ndarray:
    """Normalize's running statistics after adding the rows of x ([rows][cols]):
    a new float64 array [n, column sums, column sums of squares]."""
    x = _f64(np.atleast_2d(x))
    st = _f64(stats).copy()
    rows, cols = x.shape
    if st.shape != (1 + 2 * cols,) or lib().orc_norm_accumulate(_p(x), C.c_int64(rows), C.c_int32(cols), _p(st)):
        raise ValueError("orc_norm_accumulate rejected its arguments")
    return st


def norm_apply(stats, x, eps: float = 1e-8) -> np.ndarray:
    """x standardised with the statistics: (x - mean) / max(std, eps) per column."""
    x = _f64(np.atleast_2d(x))
    st = _f64(stats)
    rows, cols = x.shape
    out = np.empty_like(x)
    if st.shape != (1 + 2 * cols,) or lib().orc_norm_apply(_p(x), C.c_int64(rows), C.c_int32(cols), _p(st),
                                                            C.c_double(eps), _p(out)):
        raise ValueError("orc_norm_apply rejected its arguments")
    return out

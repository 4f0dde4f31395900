"""Device-side session for one partition: uploads a host-built local graph and
its inputs to HBM once, then runs the training step through the C ABI.
Argument marshalling only; the step itself runs in libmgn's kernels."""
from __future__ import annotations

import numpy as np
import torch

from . import (MGN_BF16, MGN_FP32, graph_struct, mgn_backward, mgn_create, mgn_destroy, mgn_forward,
               mgn_graph_validate, mgn_mse_grad, mgn_param_count, mgn_set_params, mgn_set_recompute,
               mgn_norm_accumulate, mgn_norm_apply, MGN_NORM_WORK_PER_COL, mgn_rollout_update, mgn_set_h1_stash,
               mgn_set_inference, mgn_sgd_step, mgn_workspace_size)


class Session:
    def __init__(self, latent: int, K: int, depth: int, precision: str, graph: dict, node_feat, edge_feat, halo,
                 params, device: str = "cuda", node_in: int = 11, edge_in: int = 4, node_out: int = 5,
                 recompute: int = 0, chunk_edges: int = 0, inference: bool = False, h1_stash: int = 0):
        """recompute: edge-stream checkpoint interval (mgn_set_recompute, bf16;
        0: keep every block); -1: the smallest interval whose workspace fits
        the device's free memory with 8 GiB to spare.  h1_stash: blocks whose
        first-Linear ReLU output the forward keeps for the backward
        (row-split kernels, mgn_set_h1_stash); -1: as many as the device's
        free memory holds beside the rest of the workspace (with 8 GiB to
        spare)."""
        if not torch.cuda.is_available():
            raise RuntimeError("libmgn needs a HIP device")
        self.device = torch.device(device)
        self.K, self.latent = K, latent
        prec = MGN_BF16 if precision == "bf16" else MGN_FP32
        self.model = mgn_create(latent, K, depth, prec, node_in, edge_in, node_out)
        dev = lambda a, dt: torch.as_tensor(np.ascontiguousarray(a, dtype=dt)).to(self.device)
        self.g = dict(n_owned=int(graph["n_owned"]), n_halo=int(graph["n_halo"]), n_edges=int(graph["n_edges"]),
                      row_ptr=dev(graph["row_ptr"], np.int32), send=dev(graph["send"], np.int32),
                      trow_ptr=dev(graph["trow_ptr"], np.int32), tedge=dev(graph["tedge"], np.int32))
        self.gs = graph_struct(self.g)
        no, nh, ne = self.g["n_owned"], self.g["n_halo"], self.g["n_edges"]
        self.node_feat = dev(np.asarray(node_feat).reshape(no, node_in), np.float32)
        self.edge_feat = dev(np.asarray(edge_feat).reshape(ne, edge_in), np.float32)
        self.halo = dev(halo, np.float32) if (nh > 0 and K > 0) else None
        self.n_params = mgn_param_count(self.model)
        self.set_params(params)
        mgn_graph_validate(self.model, self.gs)
        if recompute < 0 and not inference and K > 0 and ne > 0:
            # the smallest checkpoint interval whose workspace (as the library
            # plans it) leaves 8 GiB of the free memory: fewer blocks'
            # edge forwards repeated in the backward
            free = torch.cuda.mem_get_info(self.device)[0]
            for s in range(1, K + 1):
                mgn_set_recompute(self.model, s, chunk_edges)
                if mgn_workspace_size(self.model, self.gs) + (8 << 30) <= free:
                    recompute = s
                    break
            else:
                recompute = K
        self.recompute = max(recompute, 0)
        if self.recompute:
            mgn_set_recompute(self.model, self.recompute, chunk_edges)
        if inference:
            mgn_set_inference(self.model, True)
        self.ws_bytes = mgn_workspace_size(self.model, self.gs)
        if h1_stash < 0 and not inference and K > 0 and ne > 0:
            # the most blocks whose workspace (as the library plans it) leaves
            # 8 GiB of the free memory
            free = torch.cuda.mem_get_info(self.device)[0]
            h1_stash = 0
            for n in range(K, 0, -1):
                mgn_set_h1_stash(self.model, n)
                if mgn_workspace_size(self.model, self.gs) + (8 << 30) <= free:
                    h1_stash = n
                    break
        self.h1_stash = max(h1_stash, 0)
        mgn_set_h1_stash(self.model, self.h1_stash)
        self.ws_bytes = mgn_workspace_size(self.model, self.gs)
        self.workspace = torch.empty(max(self.ws_bytes, 256), dtype=torch.uint8, device=self.device)
        self.out = torch.empty((no, node_out), dtype=torch.float32, device=self.device)
        self.d_params = None if inference else torch.empty(self.n_params, dtype=torch.float32, device=self.device)
        self.d_halo = (torch.empty((K, nh, latent), dtype=torch.float32, device=self.device)
                       if (nh and K and not inference) else None)

    def set_params(self, params):
        if isinstance(params, torch.Tensor):
            mgn_set_params(self.model, params.to(self.device, torch.float32).contiguous())
        else:
            mgn_set_params(self.model, np.asarray(params, np.float32))

    def forward(self, stream=None):
        mgn_forward(self.model, self.gs, self.node_feat, self.edge_feat, self.halo, self.out, self.workspace, stream)
        return self.out

    def backward(self, d_out, accumulate: bool = False, stream=None):
        if not isinstance(d_out, torch.Tensor):
            d_out = torch.as_tensor(np.ascontiguousarray(d_out, np.float32)).to(self.device)
        mgn_backward(self.model, d_out.contiguous(), self.d_params, accumulate, self.d_halo, stream)
        return self.d_params, self.d_halo

    def sgd(self, lr: float, grad=None, stream=None):
        """Parameter update with the last backward's gradient (or `grad`)."""
        mgn_sgd_step(self.model, self.d_params if grad is None else grad, lr, stream)

    def rollout(self, steps: int, col0: int = 3, stream=None):
        """`steps` next-step predictions, each fed back into the flow columns
        of the node features (q <- q + p); returns the outputs of every step."""
        outs = []
        for _ in range(steps):
            self.forward(stream)
            outs.append(self.out.clone())
            mgn_rollout_update(self.out, self.node_feat, col0, stream)
        return outs

    def mse(self, target, mask=None, stream=None):
        loss = torch.empty(2, dtype=torch.float32, device=self.device)
        d_out = torch.empty_like(self.out)
        mgn_mse_grad(self.out, target, mask, loss, d_out, stream)
        return loss, d_out

    def close(self):
        """Destroys the model and drops every device buffer of the session."""
        if getattr(self, "model", None):
            mgn_destroy(self.model)
            self.model = None
        for k in ("workspace", "out", "d_params", "d_halo", "node_feat", "edge_feat", "halo", "g"):
            setattr(self, k, None)
        torch.cuda.empty_cache()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Normalizer:
    """Running per-column statistics of one kind of input (increments, node
    features or edge features) on the device, for Normalize of Algorithm 1:
    accumulate() adds rows while training, apply() standardises."""

    def __init__(self, cols: int, device: str = "cuda", eps: float = 1e-8):
        self.cols, self.eps = cols, eps
        self.stats = torch.zeros(1 + 2 * cols, dtype=torch.float64, device=device)
        self.work = torch.empty(MGN_NORM_WORK_PER_COL * cols, dtype=torch.float64, device=device)

    def accumulate(self, x, stream=None):
        mgn_norm_accumulate(x, self.stats, self.work, stream)

    def apply(self, x, out=None, stream=None):
        out = torch.empty_like(x) if out is None else out
        mgn_norm_apply(x, self.stats, out, self.eps, stream)
        return out


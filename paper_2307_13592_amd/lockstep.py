"""Several partitions of one mesh stepped in lockstep on one device: the
paper's distributed training step (Algorithm 1) with the partitions side by
side on one GPU instead of one per GPU.  One Session (model, workspace,
inputs) per part, all with the same parameters; after every block of the
forward the halo latents move from their owners into the parts that hold
them as halo, and after every block of the backward the halo gradients go
back to the owners (section "Methodology": forward halo exchange and
backward gradient exchange).  The parts' parameter gradients add up in one
buffer in part order, which takes the place of the gradient all-reduce.

Argument marshalling only: the call order lives in libmgn
(mgn_lockstep_forward / mgn_lockstep_backward), and every step, the
exchanges included, runs in its kernels."""
from __future__ import annotations

import numpy as np
import torch

from . import mgn_halo_masks, mgn_lockstep_backward, mgn_lockstep_forward, mgn_mse_grad_global, mgn_sgd_step
from .runner import Session


def nocomm_edges(send, recv, part):
    """The paper's NoComm variant (section "Results": partitions trained
    without halo exchange): only the edges whose two ends lie in the same
    part, so every part's local graph has no halo."""
    send, recv, part = (np.asarray(a, np.int32) for a in (send, recv, part))
    keep = part[send] == part[recv]
    return np.ascontiguousarray(send[keep]), np.ascontiguousarray(recv[keep])


class Lockstep:
    """P parts of one mesh; graphs[p] from mgn_graph_build(..., part, n_nodes, p),
    node_feats[p] / edge_feats[p] the part's owned-node and local-edge
    features (local order)."""

    def __init__(self, latent: int, K: int, depth: int, precision: str, part, graphs: list, node_feats: list,
                 edge_feats: list, params, device: str = "cuda", recompute: int = 0):
        self.K, self.latent, self.P = K, latent, len(graphs)
        self.device = torch.device(device)
        self.sessions = []
        for g, nf, ef in zip(graphs, node_feats, edge_feats):
            halo = np.zeros((K, g["n_halo"], latent), np.float32)  # filled by the exchange, block by block
            self.sessions.append(Session(latent, K, depth, precision, g, nf, ef, halo, params, device,
                                         recompute=recompute))
        dev = lambda a: torch.as_tensor(a).to(self.device)
        # (p, q, recv_idx, send_rows): p's halo nodes owned by q
        self.links = []
        for p, gp in enumerate(graphs):
            for q, gq in enumerate(graphs):
                if q == p or gp["n_halo"] == 0:
                    continue
                recv, send = mgn_halo_masks(gp["l2g"], gp["n_owned"], part, gq["l2g"], gq["n_owned"], q)
                if recv.size:
                    self.links.append((p, q, dev(recv), dev(send)))
        self.d_params = torch.empty(self.sessions[0].n_params, dtype=torch.float32, device=self.device)

    def forward(self, stream=None):
        """Encoders of every part; per block, the halo copies of every link,
        then the block on every part; decoders (mgn_lockstep_forward)."""
        S = self.sessions
        mgn_lockstep_forward([s.model for s in S], [s.gs for s in S], [s.node_feat for s in S],
                             [s.edge_feat for s in S], [s.halo for s in S], [s.out for s in S],
                             [s.workspace for s in S], self.links, stream)
        return [s.out for s in S]

    def mse(self, targets, masks=None, stream=None):
        """Algorithm 1's global loss: the mean squared error over the
        loss-masked owned nodes of all parts.  targets[p], masks[p] (uint8 or
        None) are device tensors of part p.  Returns (the parts' loss shares
        as device scalars, which add up to the global loss; the parts' dOut)."""
        S = self.sessions
        if masks is None:
            masks = [None] * len(S)
        rows = sum(s.out.shape[0] if m is None else int(m.count_nonzero().item()) for s, m in zip(S, masks))
        shares, d_outs = [], []
        for s, t, m in zip(S, targets, masks):
            loss = torch.empty(2, dtype=torch.float32, device=self.device)
            d_out = torch.empty_like(s.out)
            mgn_mse_grad_global(s.out, t, m, max(rows, 1), loss, d_out, stream)
            shares.append(loss[0])
            d_outs.append(d_out)
        return shares, d_outs

    def backward(self, d_outs, stream=None):
        """d_outs[p]: dL/dout of part p's owned nodes.  Returns the summed
        parameter gradient."""
        S = self.sessions
        ds = []
        for d in d_outs:
            if not isinstance(d, torch.Tensor):
                d = torch.as_tensor(np.ascontiguousarray(d, np.float32)).to(self.device)
            ds.append(d.contiguous())
        mgn_lockstep_backward([s.model for s in S], ds, self.d_params, [s.d_halo for s in S], self.links, False,
                              stream)
        return self.d_params

    def sgd(self, lr: float, stream=None):
        """Every part's model takes the same update with the summed gradient,
        so the parts' parameters stay identical."""
        for s in self.sessions:
            mgn_sgd_step(s.model, self.d_params, lr, stream)

    def close(self):
        for s in self.sessions:
            s.close()
        self.sessions = []
        self.links = []

"""A second, independent float64 formulation of the network, built from
PyTorch library layers (nn.Linear, nn.ReLU, nn.LayerNorm, index_select,
index_add_) with autograd for the gradients.  Tests only: it checks the CPU
oracle, which is written row by row without any of these.

Parameters are unpacked from the flat vector by the (name, kind, shape) list
the input generator publishes for the documented layout.
"""
from __future__ import annotations

import numpy as np
import torch
from torch import nn


def _bf16(x):
    return x.to(torch.bfloat16).to(x.dtype)


class _LinearBf16(torch.autograd.Function):
    """Linear with bfloat16 operands (mixed-precision reading): inputs and
    weights rounded for the product, the incoming gradient rounded before the
    two gradient products; bias and its gradient exact."""

    @staticmethod
    def forward(ctx, x, W, b):
        xr, Wr = _bf16(x), _bf16(W)
        ctx.save_for_backward(xr, Wr)
        return xr @ Wr.T + b

    @staticmethod
    def backward(ctx, dy):
        xr, Wr = ctx.saved_tensors
        dyr = _bf16(dy)
        return dyr @ Wr, dyr.T @ xr, dy.sum(0)


class _RoundBf16(torch.autograd.Function):
    """Storage rounding of the edge-latent stream (gradient passes through;
    the stream's own gradient is rounded by a hook on each stored tensor,
    see TorchMGN.forward)."""

    @staticmethod
    def forward(ctx, x):
        return _bf16(x)

    @staticmethod
    def backward(ctx, g):
        return g


def _apply(seq, x, bf16):
    if not bf16:
        return seq(x)
    for layer in seq:
        if isinstance(layer, nn.Linear):
            x = _LinearBf16.apply(x, layer.weight, layer.bias)
        else:
            x = layer(x)
    return x


def _mlp(fin, fout, latent, depth, ln):
    dims = [fin] + [latent] * (depth - 1) + [fout]
    layers = []
    for j in range(depth):
        layers.append(nn.Linear(dims[j], dims[j + 1]))
        if j + 1 < depth:
            layers.append(nn.ReLU())
    if ln:
        layers.append(nn.LayerNorm(fout, eps=1e-5))
    return nn.Sequential(*layers)


class TorchMGN(nn.Module):
    def __init__(self, latent, K, depth, node_in=11, edge_in=4, node_out=5, dtype=torch.float64):
        super().__init__()
        self.dtype = dtype
        self.l, self.K = latent, K
        self.enc_node = _mlp(node_in, latent, latent, depth, True)
        self.enc_edge = _mlp(edge_in, latent, latent, depth, True)
        self.edge = nn.ModuleList([_mlp(3 * latent, latent, latent, depth, True) for _ in range(K)])
        self.node = nn.ModuleList([_mlp(2 * latent, latent, latent, depth, True) for _ in range(K)])
        self.dec = _mlp(latent, node_out, latent, depth, False)
        self.to(dtype)

    def ordered_tensors(self):
        """Parameter tensors in the flat layout order."""
        out = []
        for m in [self.enc_node, self.enc_edge] + [x for k in range(self.K) for x in (self.edge[k], self.node[k])] + [self.dec]:
            for layer in m:
                if isinstance(layer, nn.Linear):
                    out += [layer.weight, layer.bias]
                elif isinstance(layer, nn.LayerNorm):
                    out += [layer.weight, layer.bias]
        return out

    def load_flat(self, flat, shapes):
        ts = self.ordered_tensors()
        assert len(ts) == len(shapes)
        off = 0
        with torch.no_grad():
            for t, (_, _, shape) in zip(ts, shapes):
                n = int(np.prod(shape))
                assert tuple(t.shape) == tuple(shape)
                t.copy_(torch.as_tensor(np.asarray(flat[off:off + n], np.float64).reshape(shape)).to(t.dtype))
                off += n
        assert off == len(flat)

    def flat_grad(self):
        return torch.cat([t.grad.reshape(-1).double() if t.grad is not None
                          else torch.zeros(t.numel(), dtype=torch.float64) for t in self.ordered_tensors()])

    def forward(self, g, node_feat, edge_feat, halo, bf16=False):
        """g: partition-local graph (row_ptr, send, n_owned, n_halo).  halo:
        tensor [K, n_halo, l] (requires_grad for d_halo)."""
        def R(x):
            if not bf16:
                return x
            y = _RoundBf16.apply(x)
            if y.requires_grad:
                # a bfloat16 tensor's gradient is bfloat16: the total gradient
                # of the stored edge latents (residual path plus MLP input)
                # is rounded once before it flows on
                y.register_hook(_bf16)
            return y
        no, nh = g["n_owned"], g["n_halo"]
        row_ptr = np.asarray(g["row_ptr"], np.int64)
        recv = torch.as_tensor(np.repeat(np.arange(no), np.diff(row_ptr)), dtype=torch.long)
        send = torch.as_tensor(np.asarray(g["send"], np.int64))
        v = _apply(self.enc_node, node_feat, bf16)
        e = R(_apply(self.enc_edge, edge_feat, bf16))
        for k in range(self.K):
            vk = torch.cat([v, halo[k]], 0) if nh > 0 else v
            m = _apply(self.edge[k], torch.cat([e, vk.index_select(0, send), vk.index_select(0, recv)], 1), bf16)
            e = R(e + m)
            agg = torch.zeros(no, self.l, dtype=self.dtype).index_add(0, recv, m)
            v = v + _apply(self.node[k], torch.cat([v, agg], 1), bf16)
        return _apply(self.dec, v, bf16)


def run(latent, K, depth, shapes, g, params, node_feat, edge_feat, halo, d_out, bf16=False,
        dtype=torch.float64):
    """Returns out, flat d_params, d_halo (numpy float64).  dtype float32 gives
    an independent single-precision implementation (used to measure how far
    a correct single-precision computation sits from the float64 oracle)."""
    torch.manual_seed(0)
    model = TorchMGN(latent, K, depth, dtype=dtype)
    model.load_flat(params, shapes)
    nf = torch.as_tensor(np.asarray(node_feat, np.float64)).to(dtype)
    ef = torch.as_tensor(np.asarray(edge_feat, np.float64)).to(dtype)
    nh = g["n_halo"]
    H = torch.as_tensor(np.asarray(halo, np.float64) if nh > 0 else np.zeros((K, 0, latent))).to(dtype)
    H = H.clone().requires_grad_(True)
    out = model(g, nf, ef, H, bf16=bf16)
    out.backward(torch.as_tensor(np.asarray(d_out, np.float64)).to(dtype))
    dh = H.grad.double().numpy() if H.grad is not None else np.zeros((K, nh, latent))
    return out.detach().double().numpy(), model.flat_grad().numpy(), dh

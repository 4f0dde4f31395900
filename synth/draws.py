"""Seeded draws: features, targets, halo latents and initial parameters.

Node input (section "Model"; 3D turbine variant of section "Results"):
  [coordinates (3), flow quantities rho,u,v,w,p (5), node-type one-hot (3)] = 11
Edge input: relative displacement sender - receiver (3) and its norm (1) = 4,
in units of the mesh's nominal cell size.  Outputs: 5 per node.
"""
from __future__ import annotations

import numpy as np

from .meshes import Mesh

NODE_IN, EDGE_IN, NODE_OUT = 11, 4, 5


def _per_block(mesh: Mesh, seed: int, what: int, width: int, fn) -> np.ndarray:
    out = np.empty((mesh.n_nodes, width), np.float64)
    for start, count, tag in mesh.stream_blocks:
        r = np.random.default_rng([seed, what, tag])
        out[start:start + count] = fn(r, (count, width))
    return out


def node_features(mesh: Mesh, seed: int) -> np.ndarray:
    """float32 [n, 11]: standardised coordinates, N(0,1) flow quantities, one-hot type."""
    c = (mesh.coords - mesh.coord_center) / mesh.coord_scale
    q = _per_block(mesh, seed, 21, 5, lambda r, s: r.standard_normal(s))
    oh = np.eye(3)[mesh.node_type.astype(np.int64)]
    return np.concatenate([c, q, oh], 1).astype(np.float32)


def edge_features(mesh: Mesh) -> np.ndarray:
    """float32 [E, 4] per directed edge s->r: (x_s - x_r)/h and |x_s - x_r|/h,
    computed in float64 and rounded once."""
    d = (mesh.coords[mesh.send] - mesh.coords[mesh.recv]) / mesh.h
    return np.concatenate([d, np.linalg.norm(d, axis=1, keepdims=True)], 1).astype(np.float32)


def targets(mesh: Mesh, seed: int) -> np.ndarray:
    """float32 [n, 5] ~ N(0, 1)."""
    return _per_block(mesh, seed, 22, NODE_OUT, lambda r, s: r.standard_normal(s)).astype(np.float32)


def halo_latents(K: int, n_halo: int, latent: int, seed: int) -> np.ndarray:
    """float32 [K, n_halo, latent] ~ N(0, 1): the halo latents handed in at the
    input of each message-passing block."""
    out = np.empty((K, n_halo, latent), np.float32)
    for k in range(K):
        out[k] = np.random.default_rng([seed, 31, k]).standard_normal((n_halo, latent), np.float32)
    return out


def param_shapes(latent: int, K: int, depth: int, node_in: int = NODE_IN,
                 edge_in: int = EDGE_IN, node_out: int = NODE_OUT) -> list[tuple[str, str, tuple]]:
    """(name, kind, shape) in flat order: EncNode, EncEdge, then per block the
    edge MLP and the node MLP, then DecNode.  Per Linear W[out][in] then b[out];
    LayerNorm gamma then beta.  Edge layer-1 inputs are [e | v_sender | v_receiver],
    node layer-1 inputs are [v | aggregated messages]."""
    out = []

    def mlp(prefix, fin, fout, ln):
        dims = [fin] + [latent] * (depth - 1) + [fout]
        for j in range(depth):
            out.append((f"{prefix}.lin{j}.W", "W", (dims[j + 1], dims[j])))
            out.append((f"{prefix}.lin{j}.b", "b", (dims[j + 1],)))
        if ln:
            out.append((f"{prefix}.ln.gamma", "gamma", (fout,)))
            out.append((f"{prefix}.ln.beta", "beta", (fout,)))

    mlp("enc_node", node_in, latent, True)
    mlp("enc_edge", edge_in, latent, True)
    for k in range(K):
        mlp(f"block{k}.edge", 3 * latent, latent, True)
        mlp(f"block{k}.node", 2 * latent, latent, True)
    mlp("dec_node", latent, node_out, False)
    return out


def perturbed(arrays, run: int, rel: float = 2.0 ** -20):
    """Copies (float64) of `arrays` with every entry scaled by 1 +- rel, the
    signs drawn from a generator seeded with (4321, run): inputs that differ
    at the level of float32 rounding, for measuring how far such noise moves
    a computation's results."""
    rng = np.random.default_rng([4321, run])
    return [None if a is None else np.asarray(a, np.float64) * (1 + rel * rng.choice([-1.0, 1.0], np.shape(a)))
            for a in arrays]


def init_params(shapes, seed: int) -> np.ndarray:
    """float32 flat: W, b ~ U(-1/sqrt(fan_in), 1/sqrt(fan_in)) (PyTorch's default
    for Linear), gamma = 1 + 0.1 N(0,1), beta = 0.1 N(0,1) (perturbed from the
    identity so the LayerNorm affine terms are exercised)."""
    r = np.random.default_rng([seed, 41])
    parts = []
    fan = None
    for name, kind, shape in shapes:
        if kind == "W":
            fan = shape[1]
            bound = 1.0 / np.sqrt(fan)
            parts.append(r.uniform(-bound, bound, shape).ravel())
        elif kind == "b":
            bound = 1.0 / np.sqrt(fan)
            parts.append(r.uniform(-bound, bound, shape).ravel())
        elif kind == "gamma":
            parts.append(1.0 + 0.1 * r.standard_normal(shape))
        else:
            parts.append(0.1 * r.standard_normal(shape))
    return np.concatenate(parts).astype(np.float32)

"""Synthetic meshes as directed COO edge lists.

Every mesh edge {a, b} appears twice, as a->b and b->a (the model's edges are
directed; section "Model" builds edge features per ordered pair).  The global
directed list is: all pairs a<b sorted by (a, b), first in the a->b direction,
then the same pairs in the b->a direction.
"""
from __future__ import annotations

from dataclasses import dataclass, field
import math

import numpy as np

NODE_NORMAL, NODE_WALL, NODE_INOUT = 0, 1, 2


@dataclass
class Mesh:
    name: str
    n_nodes: int
    send: np.ndarray          # int32 [E] global directed COO, sender
    recv: np.ndarray          # int32 [E] receiver
    coords: np.ndarray        # float64 [n, 3] physical coordinates
    h: float                  # nominal cell size (edge features are in units of h)
    node_type: np.ndarray     # int8 [n]: 0 normal, 1 wall, 2 inflow/outflow
    key: np.ndarray           # int32 [n] partition key (theta layer for sectors, 0 otherwise)
    nparts: int               # partitions the key is meant to be split into
    coord_center: np.ndarray  # frozen standardisation of node coordinates
    coord_scale: np.ndarray
    # draws are made per block of consecutive nodes so that a sub-region of a
    # mesh sees exactly the values the full mesh would: (first node, count, tag)
    stream_blocks: list = field(default_factory=list)
    part: np.ndarray | None = None   # given only for region meshes (see `sector`)

    @property
    def n_edges(self) -> int:
        return int(self.send.shape[0])


def _directed(pairs: np.ndarray) -> tuple[np.ndarray, np.ndarray]:
    """pairs: int64 [M, 2] with a < b, unique.  Returns the directed lists."""
    n = int(pairs.max()) + 1 if pairs.size else 1
    order = np.argsort(pairs[:, 0] * n + pairs[:, 1], kind="stable")
    pairs = pairs[order]
    a = pairs[:, 0].astype(np.int32)
    b = pairs[:, 1].astype(np.int32)
    return np.concatenate([a, b]), np.concatenate([b, a])


def hex_lattice(n: int = 16, name: str | None = None) -> Mesh:
    """n^3 structured hex lattice, 6-neighbour, node id = x + n*y + n*n*z."""
    idx = np.arange(n ** 3, dtype=np.int64)
    x, y, z = idx % n, (idx // n) % n, idx // (n * n)
    pairs = []
    for d, c in ((1, x), (n, y), (n * n, z)):
        a = idx[c < n - 1]
        pairs.append(np.stack([a, a + d], 1))
    send, recv = _directed(np.concatenate(pairs))
    h = 1.0 / n
    coords = np.stack([x, y, z], 1).astype(np.float64) * h
    t = np.zeros(n ** 3, np.int8)
    t[(y == 0) | (y == n - 1) | (z == 0) | (z == n - 1)] = NODE_WALL
    t[(x == 0) | (x == n - 1)] = NODE_INOUT
    ext = (n - 1) * h
    return Mesh(name or f"hex{n}", n ** 3, send, recv, coords, h, t,
                np.zeros(n ** 3, np.int32), 1,
                np.full(3, ext / 2), np.full(3, ext / 2), [(0, n ** 3, 0)])


def delaunay_box(nx: int = 50, ny: int = 50, nz: int = 40, seed: int = 2,
                 name: str | None = None) -> Mesh:
    """Cell-centred nx*ny*nz lattice in the unit box, each point jittered by
    U(-0.25, 0.25) cells per axis, tetrahedralised by Qhull's Delaunay."""
    from scipy.spatial import Delaunay

    rng = np.random.default_rng([seed, 1])
    g = np.stack(np.meshgrid(np.arange(nx), np.arange(ny), np.arange(nz), indexing="ij"), -1).reshape(-1, 3)
    hv = np.array([1.0 / nx, 1.0 / ny, 1.0 / nz])
    p = (g + 0.5 + rng.uniform(-0.25, 0.25, g.shape)) * hv
    simp = Delaunay(p).simplices.astype(np.int64)
    e = np.concatenate([simp[:, [a, b]] for a in range(4) for b in range(a + 1, 4)])
    e = np.unique(np.sort(e, 1), axis=0)
    send, recv = _directed(e)
    n = p.shape[0]
    t = np.zeros(n, np.int8)
    gx, gy, gz = g[:, 0], g[:, 1], g[:, 2]
    t[(gy == 0) | (gy == ny - 1) | (gz == 0) | (gz == nz - 1)] = NODE_WALL
    t[(gx == 0) | (gx == nx - 1)] = NODE_INOUT
    return Mesh(name or f"delaunay{nx}x{ny}x{nz}", n, send, recv, p, float(hv.max()), t,
                np.zeros(n, np.int32), 1, np.full(3, 0.5), np.full(3, 0.5), [(0, n, 0)])


# Kuhn (6-tetrahedra per cube) split of a structured lattice: its edges are the
# 3 cube edges, the 3 face diagonals e_a+e_b and the body diagonal, all taken in
# the positive index direction, so an interior node has 14 neighbours.
KUHN_DIRS = ((1, 0, 0), (0, 1, 0), (0, 0, 1), (1, 1, 0), (1, 0, 1), (0, 1, 1), (1, 1, 1))


def edge_count_sector(n_r: int, n_t: int, n_z: int) -> int:
    """Directed edge count of the full Kuhn sector mesh (closed form)."""
    return 2 * sum((n_r - a) * (n_t - b) * (n_z - c) for a, b, c in KUHN_DIRS)


def sector(n_r: int, n_t: int, n_z: int, nparts: int = 4, seed: int = 3,
           t_lo: int | None = None, t_hi: int | None = None, name: str | None = None) -> Mesh:
    """Annular, swept sector of a turbomachinery passage, n_r x n_t x n_z nodes.

    r in [0.8, 1.0], theta spans 45 degrees and is swept by 0.3 rad per unit of
    axial length, every node is jittered by U(-0.2, 0.2) cells per lattice axis.
    Node id = (j_theta * n_r + i_r) * n_z + k_z, so theta layers are contiguous
    id ranges; the partition key is the theta layer.

    With t_lo/t_hi given, only theta layers t_lo..t_hi (inclusive) are built,
    renumbered from 0 in the same order; every random draw is made per theta
    layer, so the region carries exactly the values of the full mesh.  The
    region mesh also carries `part` = theta layer // (n_t / nparts), which is
    what the slab partition of the full mesh assigns (checked by the tests).
    """
    lo = 0 if t_lo is None else max(0, t_lo)
    hi = n_t - 1 if t_hi is None else min(n_t - 1, t_hi)
    nt_loc = hi - lo + 1
    n = nt_loc * n_r * n_z
    idx = np.arange(n, dtype=np.int64)
    k = idx % n_z
    i = (idx // n_z) % n_r
    jl = idx // (n_z * n_r)
    j = jl + lo
    jit = np.empty((n, 3))
    layer = n_r * n_z
    for jj in range(lo, hi + 1):
        r = np.random.default_rng([seed, 11, jj])
        jit[(jj - lo) * layer:(jj - lo + 1) * layer] = r.uniform(-0.2, 0.2, (layer, 3))
    dth = (math.pi / 4) / (n_t - 1)
    dz = 0.9 * dth
    rad = 0.8 + 0.2 * (i + jit[:, 0]) / (n_r - 1)
    zc = dz * (k + jit[:, 2])
    th = dth * (j + jit[:, 1]) + 0.3 * zc
    coords = np.stack([rad * np.cos(th), rad * np.sin(th), zc], 1)
    t = np.zeros(n, np.int8)
    t[(i == 0) | (i == n_r - 1)] = NODE_WALL
    t[(k == 0) | (k == n_z - 1)] = NODE_INOUT
    pairs = []
    for a, b, c in KUHN_DIRS:
        ok = (i + a < n_r) & (jl + b < nt_loc) & (k + c < n_z)
        s = idx[ok]
        pairs.append(np.stack([s, s + (b * n_r + a) * n_z + c], 1))
    send, recv = _directed(np.concatenate(pairs))
    L = 0.9 * (math.pi / 4) / (n_t - 1) * (n_z - 1)
    center = np.array([0.65, 0.35, L / 2])
    scale = np.array([0.35, 0.35, L / 2])
    blocks = [((jj - lo) * layer, layer, jj) for jj in range(lo, hi + 1)]
    part = None
    if t_lo is not None or t_hi is not None:
        if n_t % nparts:
            raise ValueError("theta layers must split evenly into partitions")
        part = (j // (n_t // nparts)).astype(np.int32)
    return Mesh(name or f"sector{n_r}x{n_t}x{n_z}", n, send, recv, coords, dz, t,
                j.astype(np.int32), nparts, center, scale, blocks, part)

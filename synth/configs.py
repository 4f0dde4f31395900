"""The five benchmark configurations and small variants used by the tests.

C1  16^3 hex lattice (4,096 nodes, 23,040 directed edges), l=64,  K=2,  D=2, fp32
C2  100k-point jittered Delaunay box (~1.55M directed edges), l=128, K=15, D=2, fp32
C3  sector 50x160x500, partition 1 of 4 theta slabs (1M owned, 50k halo), l=128, K=15, D=2, fp32
C4  sector 100x160x500, partition 1 of 4 (2M owned, 100k halo), l=128, K=15, D=2, bf16
C5  sector 100x160x1000, partition 1 of 4 (4M owned, 200k halo), l=256, K=15, D=3, bf16
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Callable

import numpy as np

from . import meshes, draws


@dataclass
class Config:
    name: str
    build_mesh: Callable[[bool], meshes.Mesh]   # arg: region-only (sector meshes)
    part: int            # which partition is run (0 with one partition)
    latent: int
    K: int
    depth: int
    precision: str       # "fp32" or "bf16"
    seed: int
    note: str = ""


def _sector_cfg(n_r, n_t, n_z, nparts, seed, p):
    L = n_t // nparts

    def build(region: bool):
        if region:
            return meshes.sector(n_r, n_t, n_z, nparts, seed, t_lo=p * L - 1, t_hi=(p + 1) * L)
        return meshes.sector(n_r, n_t, n_z, nparts, seed)
    return build


CONFIGS: dict[str, Config] = {
    "C1": Config("C1", lambda region: meshes.hex_lattice(16), 0, 64, 2, 2, "fp32", 1,
                 "16^3 hex lattice, 6-neighbour"),
    "C2": Config("C2", lambda region: meshes.delaunay_box(50, 50, 40, seed=2), 0, 128, 15, 2, "fp32", 2,
                 "Delaunay of 100k jittered points in the unit box"),
    "C3": Config("C3", _sector_cfg(50, 160, 500, 4, 3, 1), 1, 128, 15, 2, "fp32", 3,
                 "sector 50x160x500, theta slab 1 of 4"),
    "C4": Config("C4", _sector_cfg(100, 160, 500, 4, 4, 1), 1, 128, 15, 2, "bf16", 4,
                 "sector 100x160x500, theta slab 1 of 4"),
    "C5": Config("C5", _sector_cfg(100, 160, 1000, 4, 5, 1), 1, 256, 15, 3, "bf16", 5,
                 "sector 100x160x1000, theta slab 1 of 4"),
}


def small_sector(n_r=6, n_t=16, n_z=10, nparts=4, p=1, latent=64, K=3, depth=2,
                 precision="fp32", seed=7, region=False) -> Config:
    return Config(f"sector{n_r}x{n_t}x{n_z}_p{p}_l{latent}K{K}D{depth}{precision}",
                  _sector_cfg(n_r, n_t, n_z, nparts, seed, p), p, latent, K, depth, precision, seed)


@dataclass
class Case:
    """Global inputs of one configuration (before the partition-local build)."""
    cfg: Config
    mesh: meshes.Mesh
    node_feat: np.ndarray     # float32 [n, 11]
    edge_feat: np.ndarray     # float32 [E, 4] in global directed order
    target: np.ndarray        # float32 [n, 5]
    params: np.ndarray        # float32 [P]
    shapes: list = field(default_factory=list)

    def local_inputs(self, l2g: np.ndarray, eperm: np.ndarray, n_owned: int, n_halo: int) -> dict:
        """Inputs in a partition-local order (owned rows by local id, edges in
        receiver-sorted local order, halo latents in local halo order)."""
        c = self.cfg
        return dict(
            node_feat=np.ascontiguousarray(self.node_feat[l2g[:n_owned]]),
            edge_feat=np.ascontiguousarray(self.edge_feat[eperm]),
            target=np.ascontiguousarray(self.target[l2g[:n_owned]]),
            halo=draws.halo_latents(c.K, n_halo, c.latent, c.seed),
        )


def make_case(cfg: Config, region: bool = True) -> Case:
    mesh = cfg.build_mesh(region)
    shapes = draws.param_shapes(cfg.latent, cfg.K, cfg.depth)
    return Case(cfg, mesh, draws.node_features(mesh, cfg.seed), draws.edge_features(mesh),
                draws.targets(mesh, cfg.seed), draws.init_params(shapes, cfg.seed), shapes)

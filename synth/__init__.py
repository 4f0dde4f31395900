"""Seeded synthetic inputs for the MeshGraphNets training step.

This package only *draws* inputs: meshes (directed COO edge lists), node and
edge features, targets, halo latents and initial parameters.  It holds none of
the network's arithmetic, so both the CPU oracle and the GPU library can be fed
from it without sharing any of the computation they are compared on.

The meshes stand in for the paper's datasets (the public 2D cylinder flow set
and the proprietary 3D turbine stator, section "Results"), which are not
available: a structured hex lattice, a jittered Delaunay tetra mesh in a box,
and an annular, swept turbomachinery-like sector split into a Kuhn tetra mesh
and partitioned into theta slabs (the stand-in for the METIS partition of
section "Methodology").
"""
from .meshes import Mesh, hex_lattice, delaunay_box, sector, edge_count_sector
from .draws import node_features, edge_features, targets, halo_latents, init_params, param_shapes, perturbed
from .configs import CONFIGS, Config, make_case, Case

__all__ = [
    "Mesh", "hex_lattice", "delaunay_box", "sector", "edge_count_sector",
    "node_features", "edge_features", "targets", "halo_latents", "init_params", "param_shapes", "perturbed",
    "CONFIGS", "Config", "make_case", "Case",
]

"""Operation and memory counts of the convolution schemes (reports only).

Per input-output channel pair and leaf of edge s:
- naive: the 3^3 kernel at every voxel of the cell, 27 s^3 products;
- truncated (the supplement's efficient convolution): the kernel once on the
  cell's constant value, plus, at every boundary voxel, the taps that leave
  the cell (19 at a corner, 15 along an edge, 9 on a face): for s = 8 that
  is 27 + 8*19 + 12*6*15 + 6*6^2*9 = 3203;
- window sums: 27 products against the 27 window sums of the leaf (the sums
  themselves are additions), for every s.
"""
from __future__ import annotations


def outside_taps(s: int) -> int:
    """Taps of the cell's boundary voxels that reach outside an s^3 cell."""
    if s == 1:
        return 26
    return 8 * 19 + 12 * (s - 2) * 15 + 6 * (s - 2) ** 2 * 9


def conv_products(s: int, scheme: str) -> int:
    if scheme == "naive":
        return 27 * s ** 3
    if scheme == "truncated":
        return 27 + outside_taps(s)
    if scheme == "window_sums":
        return 27
    raise ValueError(scheme)


def workload_products(leaves_by_edge: dict, cin: int, cout: int) -> dict:
    """Products of one conv layer over a leaf-size histogram {edge: count}."""
    return {sch: cin * cout * sum(n * conv_products(s, sch) for s, n in leaves_by_edge.items())
            for sch in ("naive", "truncated", "window_sums")}


def octree_bytes(n_trees: int, n_leaves: int, c: int) -> int:
    """Bit strings (16 B) and prefix (8 B) per tree, c floats per leaf."""
    return 24 * n_trees + 4 * c * n_leaves


def dense_bytes(voxels: int, c: int) -> int:
    return 4 * c * voxels

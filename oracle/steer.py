"""Feature-Steering of a sparse tensor by a rigid motion (oracle; test infrastructure only).

Sec. 4.1: the features F_n are rotated by rho(r), the block-diagonal matrix of the Wigner-D
matrices of the feature's irreducible fields (Eq. 5), applied by a matrix product; the sites
H_n are converted to real-world point coordinates, moved by (r, t) and re-voxelised, and sites
that land in one cell are merged with their features averaged.

Readings where the paper is silent:
  * the real-world point of site x is the centre of its cell, origin + (x + 1/2) * voxel per
    axis (the cell convention of the voxelisation oracle), and the moved point is r p + t;
  * that centre and the moved point are computed in fp32 in the order
    ((r_a0 p_0 + r_a1 p_1) + r_a2 p_2) + t_a, each product and sum rounded to nearest (no fused
    multiply-add), from r, t, origin and voxel rounded to fp32, because they decide the integer
    cells; the new cells, the dropping of points outside the grid and the lexicographic site
    order are the voxelisation's;
  * the rotated features are averaged over merged sites in fp64 (the mean of rotated features
    equals the rotation of the mean features).
"""
import numpy as np

from . import sh
from . import voxel as ov


def site_points(coords: np.ndarray, origin, voxel: float) -> np.ndarray:
    """fp32 cell centres origin + (x + 1/2) voxel of sites (b, x, y, z) -> [n, 3]."""
    c = np.asarray(coords, np.int64).reshape(-1, 4)[:, 1:]
    o = np.asarray(origin, np.float32).reshape(3)
    return (c.astype(np.float32) + np.float32(0.5)) * np.float32(voxel) + o


def moved_points(points: np.ndarray, R: np.ndarray, t) -> np.ndarray:
    """fp32 r p + t with the operation order stated above."""
    p = np.asarray(points, np.float32)
    r = np.asarray(R, np.float64).astype(np.float32)
    tt = np.asarray(t, np.float64).astype(np.float32)
    out = np.empty_like(p)
    for a in range(3):
        out[:, a] = ((r[a, 0] * p[:, 0] + r[a, 1] * p[:, 1]) + r[a, 2] * p[:, 2]) + tt[a]
    return out


def steer(coords: np.ndarray, feats: np.ndarray, fields, R: np.ndarray, t, origin, voxel: float, grid):
    """Returns (coords' int32 [m, 4], feats' fp64 [m, C], site_row [n]: the new row of each input
    site or -1 when it left the grid)."""
    c = np.asarray(coords, np.int32).reshape(-1, 4)
    f = np.asarray(feats, np.float64).reshape(len(c), -1)
    rho = sh.block_rep(fields, np.asarray(R, np.float64))
    rotated = f @ rho.T
    p = moved_points(site_points(c, origin, voxel), R, t)
    return ov.voxelize(p, c[:, 0], rotated, origin, voxel, grid)

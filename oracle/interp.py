"""Tensor-to-Point: trilinear interpolation of a sparse tensor at points, and its adjoint
(oracle; test infrastructure only).

Sec. 4.1 interpolates point-wise features from the sparse backbone maps (the module is cited,
not specified).  Reading taken here: the features live at the cell centres
origin + (x + 1/2) voxel of the active sites and are zero elsewhere; a point p is interpolated
trilinearly between the 8 site centres around it, i.e. the value at p of the trilinear
interpolant of the zero-filled grid.  With u = (p - origin) / voxel - 1/2 per axis (computed in
fp32 in that order, because floor(u) decides which sites are read), x0 = floor(u) and
w = u - x0, corner x0 + c (c in {0, 1}^3) has weight prod_a (c_a ? w_a : 1 - w_a).  Corners
outside the grid or inactive contribute nothing; sites of other batch entries are never read.
The backward pass is the exact adjoint: every point scatters weight * grad to its corners.
Arithmetic after the fp32 cell decision is fp64.
"""
import numpy as np


def point_corners(points: np.ndarray, origin, voxel: float):
    """(x0 int64 [n, 3], w fp64 [n, 3]) from the fp32 u = (p - origin) / voxel - 1/2."""
    p = np.asarray(points, np.float32).reshape(-1, 3)
    o = np.asarray(origin, np.float32).reshape(3)
    u = (p - o) / np.float32(voxel) - np.float32(0.5)
    x0 = np.floor(u)
    with np.errstate(invalid="ignore"):      # non-finite points: their corners are never read
        return np.where(np.isfinite(x0), x0, 0).astype(np.int64), (u.astype(np.float64) - x0.astype(np.float64))


def corner_table(coords, points, batch, origin, voxel: float):
    """[n, 8] site row of each corner (-1 if inactive) and [n, 8] weights, corner c = (cx, cy, cz)
    at index 4 cx + 2 cy + cz."""
    H = {tuple(int(v) for v in c): r for r, c in enumerate(np.asarray(coords, np.int64))}
    x0, w = point_corners(points, origin, voxel)
    n = len(x0)
    b = np.zeros(n, np.int64) if batch is None else np.asarray(batch, np.int64)
    rows = np.full((n, 8), -1, np.int64)
    wts = np.zeros((n, 8))
    for i in range(n):
        if not np.all(np.isfinite(w[i])):
            continue
        for k in range(8):
            c = ((k >> 2) & 1, (k >> 1) & 1, k & 1)
            wts[i, k] = np.prod([w[i, a] if c[a] else 1.0 - w[i, a] for a in range(3)])
            rows[i, k] = H.get((int(b[i]), int(x0[i, 0] + c[0]), int(x0[i, 1] + c[1]), int(x0[i, 2] + c[2])), -1)
    return rows, wts


def interpolate(coords, feats, points, batch, origin, voxel: float) -> np.ndarray:
    rows, wts = corner_table(coords, points, batch, origin, voxel)
    F = np.asarray(feats, np.float64)
    out = np.zeros((len(rows), F.shape[1]))
    for k in range(8):
        m = rows[:, k] >= 0
        out[m] += wts[m, k, None] * F[rows[m, k]]
    return out


def interpolate_backward(coords, n_sites: int, points, batch, grad, origin, voxel: float) -> np.ndarray:
    rows, wts = corner_table(coords, points, batch, origin, voxel)
    g = np.asarray(grad, np.float64)
    dF = np.zeros((n_sites, g.shape[1]))
    for k in range(8):
        m = rows[:, k] >= 0
        np.add.at(dF, rows[m, k], wts[m, k, None] * g[m])
    return dF

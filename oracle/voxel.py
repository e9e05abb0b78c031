"""Voxelisation of point clouds with per-cell feature averaging (oracle; test infrastructure only).

Sec. 4.1: a site is active when the grid cell of that site encloses any input point, and the
site's feature is the average of the features of the points its cell encloses (the paper's
points carry (R, G, B, 1)).  Feature-Steering (Sec. 4.1) re-voxelises transformed sites the same
way, merging sites that land in one cell and averaging their features.

Readings where the paper is silent:
  * the cell of site x = (x, y, z) is [origin + x*voxel, origin + (x+1)*voxel) per axis, so a
    point p belongs to floor((p - origin) / voxel); the subtraction and the division are taken
    in fp32 (the precision of the inputs), which decides the integer cell exactly;
  * points whose cell lies outside [0, grid) (or whose coordinates are not finite) are dropped;
  * every point carries a batch index b in [0, nbatch); cells never merge across b;
  * sites are listed in lexicographic (b, x, y, z) order, like every generated site set;
  * the average is the plain mean over the cell's points (fp64 here).

Everything but the cell decision is fp64 numpy.
"""
import numpy as np


def point_cells(points: np.ndarray, origin, voxel: float, grid) -> np.ndarray:
    """[n, 3] int64 cell of every point (fp32 arithmetic), -1 rows for dropped points."""
    p = np.asarray(points, np.float32).reshape(-1, 3)
    o = np.asarray(origin, np.float32).reshape(3)
    t = (p - o) / np.float32(voxel)                      # fp32, correctly rounded
    g = np.asarray(grid, np.int64).reshape(3) if np.ndim(grid) else np.full(3, int(grid))
    with np.errstate(invalid="ignore"):
        keep = np.all((t >= 0) & (t < g.astype(np.float32)), axis=1)
    cells = np.full((len(p), 3), -1, np.int64)
    cells[keep] = np.floor(t[keep]).astype(np.int64)   # 0 <= t < g, so 0 <= floor(t) < g
    return cells


def voxelize(points: np.ndarray, batch: np.ndarray, feats: np.ndarray, origin, voxel: float, grid):
    """Returns (coords int32 [m, 4] as (b, x, y, z) lexicographic, averaged features [m, C] fp64,
    point_row int64 [n]: the site row of each point or -1)."""
    cells = point_cells(points, origin, voxel, grid)
    n = len(cells)
    b = np.zeros(n, np.int64) if batch is None else np.asarray(batch, np.int64).reshape(n)
    f = np.asarray(feats, np.float64)
    f = f.reshape(n, f.shape[-1] if f.ndim == 2 else 1)
    sums, counts = {}, {}
    for i in range(n):
        if cells[i, 0] < 0:
            continue
        key = (int(b[i]), int(cells[i, 0]), int(cells[i, 1]), int(cells[i, 2]))
        if key in sums:
            sums[key] += f[i]
            counts[key] += 1
        else:
            sums[key] = f[i].copy()
            counts[key] = 1
    keys = sorted(sums)
    row = {k: r for r, k in enumerate(keys)}
    coords = np.array(keys, np.int32).reshape(-1, 4)
    out = np.array([sums[k] / counts[k] for k in keys], np.float64).reshape(len(keys), f.shape[1])
    point_row = np.full(n, -1, np.int64)
    for i in range(n):
        if cells[i, 0] >= 0:
            point_row[i] = row[(int(b[i]), int(cells[i, 0]), int(cells[i, 1]), int(cells[i, 2]))]
    return coords, out, point_row

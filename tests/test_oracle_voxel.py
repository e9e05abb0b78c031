"""Pins for the oracle's voxelisation with per-cell feature averaging (Sec. 4.1).

The cell test of the paper (the grid cell of a site encloses the point) is checked by brute
force over every cell of small grids, in exact arithmetic on dyadic coordinates (exactly
representable, so the fp32 cell decision cannot differ); the averages are checked against
per-cell sums taken directly from that enumeration.  Invariants: feature conservation
(count x mean summed over sites equals the sum over kept points), the constant channel
averages to exactly 1, invariance to the order of the points, equivariance to shifts by whole
voxels, no merging across batch entries, boundary and non-finite points.
"""
from fractions import Fraction

import numpy as np

from oracle import voxel as ov


def _dyadic_cloud(rng, n, grid, origin, vox, denom=64):
    """Points on a 1/denom lattice spanning slightly more than the grid (some fall outside)."""
    lo = origin - vox
    span = (grid + 2) * vox
    q = rng.integers(0, int(span * denom), size=(n, 3))
    return (lo + q / denom).astype(np.float32)


def test_cells_and_means_by_bruteforce():
    rng = np.random.default_rng(20211107)
    grid, origin, vox = 5, -1.0, 0.5
    pts = _dyadic_cloud(rng, 300, grid, origin, vox)
    b = rng.integers(0, 2, size=300)
    f = rng.standard_normal((300, 3))
    coords, mean, row = ov.voxelize(pts, b, f, (origin,) * 3, vox, grid)
    # brute force: every (b, cell) of the grid, membership by exact comparison
    want_keys, want_mean = [], []
    P = [[Fraction(float(v)) for v in p] for p in pts]
    o, v = Fraction(origin), Fraction(vox)
    for bb in range(2):
        for x in range(grid):
            for y in range(grid):
                for z in range(grid):
                    lo = [o + c * v for c in (x, y, z)]
                    members = [i for i in range(len(P)) if b[i] == bb and
                               all(lo[a] <= P[i][a] < lo[a] + v for a in range(3))]
                    if members:
                        want_keys.append((bb, x, y, z))
                        want_mean.append(f[members].sum(0) / len(members))
    np.testing.assert_array_equal(coords, np.array(want_keys, np.int32))
    np.testing.assert_allclose(mean, np.array(want_mean), rtol=1e-13, atol=1e-13)
    for i in range(len(P)):
        if row[i] >= 0:
            assert tuple(coords[row[i]]) in set(want_keys)
            c = coords[row[i]]
            assert c[0] == b[i] and all(o + c[1 + a] * v <= P[i][a] < o + (c[1 + a] + 1) * v for a in range(3))


def test_conservation_constant_channel_and_permutation():
    rng = np.random.default_rng(5)
    pts = rng.uniform(-2.0, 34.0, size=(5000, 3)).astype(np.float32)
    b = rng.integers(0, 3, size=5000)
    rgb = rng.uniform(0, 1, size=(5000, 3))
    f = np.concatenate([rgb, np.ones((5000, 1))], 1)       # (R, G, B, 1) as in Sec. 4.1
    coords, mean, row = ov.voxelize(pts, b, f, (0.0, 0.0, 0.0), 1.0, 32)
    kept = row >= 0
    counts = np.bincount(row[kept], minlength=len(coords))
    assert counts.min() >= 1
    np.testing.assert_allclose((counts[:, None] * mean).sum(0), f[kept].sum(0), rtol=1e-12)
    assert np.all(mean[:, 3] == 1.0)
    assert np.all(np.diff(coords.astype(np.int64) @ np.array([1 << 30, 1 << 20, 1 << 10, 1])) > 0)  # lexicographic
    perm = rng.permutation(5000)
    c2, m2, r2 = ov.voxelize(pts[perm], b[perm], f[perm], (0.0, 0.0, 0.0), 1.0, 32)
    np.testing.assert_array_equal(c2, coords)
    np.testing.assert_allclose(m2, mean, rtol=1e-12, atol=1e-12)
    np.testing.assert_array_equal(r2, row[perm])


def test_shift_by_whole_voxels():
    rng = np.random.default_rng(9)
    pts = (rng.integers(0, 20 * 16, size=(800, 3)) / 16.0).astype(np.float32)   # inside [0, 20)
    f = rng.standard_normal((800, 2))
    c0, m0, _ = ov.voxelize(pts, None, f, (0.0, 0.0, 0.0), 1.0, 32)
    t = np.array([3, 7, 1])
    c1, m1, _ = ov.voxelize(pts + t.astype(np.float32), None, f, (0.0, 0.0, 0.0), 1.0, 32)
    np.testing.assert_array_equal(c1[:, 1:], c0[:, 1:] + t)
    np.testing.assert_allclose(m1, m0, rtol=1e-14)


def test_boundaries_batches_and_nonfinite():
    pts = np.array([[0.0, 0.0, 0.0],      # lower face of cell 0: inside
                    [1.0, 0.5, 0.5],      # lower face of cell 1 in x
                    [3.999, 0.0, 0.0],    # last cell
                    [4.0, 0.0, 0.0],      # upper grid bound: dropped
                    [-1e-6, 0.0, 0.0],    # just below the grid: dropped
                    [np.nan, 0.0, 0.0],   # not finite: dropped
                    [0.25, 0.25, 0.25],   # same cell as point 0, same batch: merged
                    [0.25, 0.25, 0.25]],  # same position, other batch: its own site
                   np.float32)
    b = np.array([0, 0, 0, 0, 0, 0, 0, 1])
    f = np.arange(8, dtype=np.float64)[:, None]
    coords, mean, row = ov.voxelize(pts, b, f, (0.0, 0.0, 0.0), 1.0, 4)
    np.testing.assert_array_equal(coords, [[0, 0, 0, 0], [0, 1, 0, 0], [0, 3, 0, 0], [1, 0, 0, 0]])
    np.testing.assert_array_equal(row, [0, 1, 2, -1, -1, -1, 0, 3])
    np.testing.assert_array_equal(mean[:, 0], [(0 + 6) / 2, 1, 2, 7])

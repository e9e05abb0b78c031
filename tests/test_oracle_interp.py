"""Pins for the oracle's Tensor-to-Point interpolation (Sec. 4.1).

* It equals scipy's order-1 (trilinear) map_coordinates of the zero-filled dense grid, sampled
  at the same continuous voxel coordinates, for points anywhere in the grid (an independent
  implementation of the same definition).
* At a site centre it returns that site's features exactly; with all 8 corners active and
  constant features it returns the constant (partition of unity).
* The backward pass is the adjoint: <interp(F), g> = <F, interp*(g)>.
"""
import numpy as np
from scipy import ndimage

from oracle import interp as oi


def _sites(rng, n, grid):
    c = np.stack([np.zeros(n, int)] + [rng.integers(0, grid, n) for _ in range(3)], 1)
    return np.unique(c, axis=0).astype(np.int32)


def test_matches_dense_trilinear():
    rng = np.random.default_rng(1)
    grid, origin, vox = 10, np.array([-1.0, 0.5, 2.0]), 0.5
    c = _sites(rng, 400, grid)
    f = rng.standard_normal((len(c), 3))
    pts = (origin + rng.uniform(0, grid * vox, (500, 3))).astype(np.float32)
    got = oi.interpolate(c, f, pts, None, origin, vox)
    dense = np.zeros((3, grid, grid, grid))
    dense[:, c[:, 1], c[:, 2], c[:, 3]] = f.T
    u = (pts.astype(np.float32) - origin.astype(np.float32)) / np.float32(vox) - np.float32(0.5)
    for ch in range(3):
        want = ndimage.map_coordinates(dense[ch], u.T.astype(np.float64), order=1, mode="grid-constant", cval=0.0)
        np.testing.assert_allclose(got[:, ch], want, atol=1e-12)


def test_site_centres_and_partition_of_unity():
    rng = np.random.default_rng(2)
    c = _sites(rng, 300, 8)
    f = rng.standard_normal((len(c), 4))
    centres = (c[:, 1:] + 0.5).astype(np.float32)
    np.testing.assert_allclose(oi.interpolate(c, f, centres, None, (0.0, 0.0, 0.0), 1.0), f, atol=1e-15)
    xyz = np.stack(np.meshgrid(*[np.arange(8)] * 3, indexing="ij"), -1).reshape(-1, 3)
    full = np.concatenate([np.zeros((512, 1), int), xyz], 1).astype(np.int32)
    const = np.tile([[2.5, -1.0]], (512, 1))
    pts = rng.uniform(0.5, 7.5, (200, 3)).astype(np.float32)
    np.testing.assert_allclose(oi.interpolate(full, const, pts, None, (0.0, 0.0, 0.0), 1.0),
                               np.tile([[2.5, -1.0]], (200, 1)), atol=1e-12)


def test_adjoint_identity_and_batches():
    rng = np.random.default_rng(3)
    c = np.concatenate([_sites(rng, 200, 8), _sites(rng, 200, 8) + np.array([1, 0, 0, 0], np.int32)])
    f = rng.standard_normal((len(c), 3))
    pts = rng.uniform(-1, 9, (300, 3)).astype(np.float32)
    b = rng.integers(0, 2, 300)
    g = rng.standard_normal((300, 3))
    lhs = (oi.interpolate(c, f, pts, b, (0.0, 0.0, 0.0), 1.0) * g).sum()
    rhs = (f * oi.interpolate_backward(c, len(c), pts, b, g, (0.0, 0.0, 0.0), 1.0)).sum()
    assert abs(lhs - rhs) <= 1e-12 * max(1.0, abs(lhs))
    # a point never reads sites of another batch entry
    only0 = oi.interpolate(c, np.where((c[:, 0] == 0)[:, None], f, 0.0), pts, b, (0.0, 0.0, 0.0), 1.0)
    assert np.all(only0[b == 1] == 0.0)

"""GPU parity of the voxelisation with per-cell feature averaging (Sec. 4.1) against the oracle.

Sites and the site row of every point must match exactly (the cell decision is taken in fp32 on
both sides); averaged features within 1e-4 (L_inf error over the L_inf norm), the constant
channel exactly 1.  Every call goes through the C ABI.
"""
import numpy as np
import pytest

from cases import rel_err
from oracle import voxel as ov
from workloads import CONFIGS
from workloads.gen import make_point_cloud

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
P = pytest.importorskip("paper_2111_07383_amd")
from paper_2111_07383_amd import _abi  # noqa: E402

DEV = "cuda:0"


def _run(points, batch, feats, nbatch, origin, voxel, grid):
    pt = torch.from_numpy(np.ascontiguousarray(points, np.float32)).to(DEV)
    bt = None if batch is None else torch.from_numpy(np.ascontiguousarray(batch, np.int32)).to(DEV)
    ft = None if feats is None else torch.from_numpy(np.ascontiguousarray(feats, np.float32)).to(DEV)
    c, f, r = P.voxelize(pt, ft, bt, nbatch, origin, voxel, grid)
    return c.cpu().numpy(), (None if f is None else f.cpu().numpy()), r.cpu().numpy()


def _check(points, batch, feats, nbatch, origin, voxel, grid):
    c, f, r = _run(points, batch, feats, nbatch, origin, voxel, grid)
    wc, wf, wr = ov.voxelize(points, batch, feats if feats is not None else np.zeros((len(points), 0)),
                             origin, voxel, grid)
    np.testing.assert_array_equal(c, wc)
    np.testing.assert_array_equal(r, wr)
    if feats is not None and len(wc):
        assert rel_err(f, wf) < 1e-4
    return c, f, r


def test_object_clouds_rgb1():
    """The benchmark's 32 object clouds (524 288 points, some outside the grid)."""
    points, batch, feats = make_point_cloud(CONFIGS[7])
    print(f"voxelise {len(points)} points", flush=True)
    c, f, r = _check(points, batch, feats, 32, (0.0, 0.0, 0.0), 1.0, 64)
    assert np.all(f[:, 3] == 1.0) and (r < 0).any()


@pytest.mark.parametrize("n,C,grid,voxel,origin,nbatch", [
    (1, 3, 8, 1.0, (0.0, 0.0, 0.0), 1),
    (7, 1, (5, 6, 7), 0.5, (-1.0, -1.5, 0.25), 2),        # ragged, anisotropic grid
    (5000, 4, 16, 0.37, (-0.3, 0.1, -2.0), 3),             # voxel not a power of two
    (20000, 0, 32, 1.0, (0.0, 0.0, 0.0), 4),               # coordinates only
    (3000, 2, 4, 8.0, (0.0, 0.0, 0.0), 1),                 # many points per cell
    (2000, 3, 2, 16.0, (0.0, 0.0, 0.0), 1),                # hundreds per cell: the workgroup sort in LDS
    (20000, 2, 2, 16.0, (0.0, 0.0, 0.0), 1),               # ~2500 per cell: LDS sort of up to 8192 entries
    (60000, 1, 1, 40.0, (0.0, 0.0, 0.0), 1),               # ~60 000 in one cell: the sort in global memory
])
def test_random_clouds(n, C, grid, voxel, origin, nbatch):
    rng = np.random.default_rng(n + C)
    g = np.asarray(grid if np.ndim(grid) else (grid,) * 3, np.float64)
    lo = np.asarray(origin) - voxel
    pts = (lo + rng.uniform(0, 1, (n, 3)) * (g + 2) * voxel).astype(np.float32)
    batch = rng.integers(0, nbatch, n).astype(np.int32)
    feats = rng.standard_normal((n, C)).astype(np.float32) if C else None
    print(f"voxelise n={n} C={C} grid={grid}", flush=True)
    _check(pts, batch, feats, nbatch, origin, voxel, grid)


def test_edges_and_errors():
    pts = np.array([[0.0, 0.0, 0.0], [4.0, 0.0, 0.0], [np.nan, 1.0, 1.0], [np.inf, 1.0, 1.0],
                    [0.5, 0.5, 0.5], [3.5, 3.5, 3.5]], np.float32)
    feats = np.arange(12, dtype=np.float32).reshape(6, 2)
    c, f, r = _check(pts, None, feats, 1, (0.0, 0.0, 0.0), 1.0, 4)
    np.testing.assert_array_equal(r, [0, -1, -1, -1, 0, 1])
    # every point outside: no sites
    c, f, r = _run(pts[1:4], None, feats[1:4], 1, (0.0, 0.0, 0.0), 1.0, 4)
    assert len(c) == 0 and np.all(r == -1)
    # no points
    c, f, r = _run(np.zeros((0, 3), np.float32), None, np.zeros((0, 2), np.float32), 1, (0.0, 0.0, 0.0), 1.0, 4)
    assert len(c) == 0 and len(r) == 0
    # a batch index outside [0, nbatch)
    with pytest.raises(_abi.SSConvError) as e:
        _run(pts, np.array([0, 0, 0, 0, 2, 0], np.int32), feats, 2, (0.0, 0.0, 0.0), 1.0, 4)
    assert e.value.code == _abi.E_BOUNDS
    with pytest.raises(_abi.SSConvError) as e:
        _run(pts, None, feats, 1, (0.0, 0.0, 0.0), 0.0, 4)
    assert e.value.code == _abi.E_INVALID


def test_voxelize_deterministic():
    points, batch, feats = make_point_cloud(CONFIGS[7])
    a = _run(points, batch, feats, 32, (0.0, 0.0, 0.0), 1.0, 64)
    b = _run(points, batch, feats, 32, (0.0, 0.0, 0.0), 1.0, 64)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)

"""GPU parity of Feature-Steering (Sec. 4.1) against the oracle: new sites and the new row of
every input site exact (the moved cell centres are computed in fp32 in the same order on both
sides), steered features within 1e-4 (L_inf error over the L_inf norm).  Through the C ABI.
"""
import numpy as np
import pytest

from cases import rel_err
from oracle import sh
from oracle import steer as ost
from workloads import CONFIGS
from workloads.gen import make_coords, make_features, make_motion

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
P = pytest.importorskip("paper_2111_07383_amd")
from paper_2111_07383_amd import _abi  # noqa: E402

DEV = "cuda:0"
F_SMALL = ((0, 2), (1, 2), (2, 1), (3, 1), (4, 1))   # every order the library supports: 29 channels


def _check(coords, feats, fields, R, t, nbatch, origin, voxel, grid):
    ct = torch.from_numpy(np.ascontiguousarray(coords, np.int32)).to(DEV)
    ft = torch.from_numpy(np.ascontiguousarray(feats, np.float32)).to(DEV)
    c, f, r = P.steer(ct, ft, fields, R, t, nbatch, origin, voxel, grid)
    wc, wf, wr = ost.steer(coords, feats, fields, R, t, origin, voxel, grid)
    np.testing.assert_array_equal(c.cpu().numpy(), wc)
    np.testing.assert_array_equal(r.cpu().numpy(), wr)
    if len(wc):
        err = rel_err(f.cpu().numpy(), wf)
        print(f"steer: {len(coords)} -> {len(wc)} sites, feature error {err:.2e}", flush=True)
        assert err < 1e-4
    return c, f, r


def test_steer_backbone_map():
    """The benchmark's 64^3 map with 104 channels of orders 0, 1, 2 under its seeded motion."""
    spec = CONFIGS[8]
    coords = make_coords(spec)
    feats = make_features(spec, len(coords), spec.layers[0].cin)
    R, t = make_motion(spec)
    _check(coords, feats, spec.layers[0].fields_in, R, t, 1, (0.0, 0.0, 0.0), 1.0, spec.grid)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_steer_random_motions_all_orders(seed):
    rng = np.random.default_rng(100 + seed)
    c = np.stack([rng.integers(0, 3, 2000)] + [rng.integers(0, 24, 2000) for _ in range(3)], 1)
    coords = np.unique(c, axis=0).astype(np.int32)
    feats = rng.standard_normal((len(coords), 29)).astype(np.float32)
    q = rng.standard_normal(4)
    q /= np.linalg.norm(q)
    w, x, y, z = q
    R = np.array([[1 - 2 * (y * y + z * z), 2 * (x * y - z * w), 2 * (x * z + y * w)],
                  [2 * (x * y + z * w), 1 - 2 * (x * x + z * z), 2 * (y * z - x * w)],
                  [2 * (x * z - y * w), 2 * (y * z + x * w), 1 - 2 * (x * x + y * y)]])
    t = rng.uniform(-3, 3, 3)
    _check(coords, feats, F_SMALL, R, t, 3, (-1.0, 0.5, -0.25), 0.75, 24)


def test_steer_cube_rotation_and_identity():
    rng = np.random.default_rng(7)
    c = np.stack([np.zeros(500, int)] + [rng.integers(2, 14, 500) for _ in range(3)], 1)
    coords = np.unique(c, axis=0).astype(np.int32)
    feats = rng.standard_normal((len(coords), 29)).astype(np.float32)
    _, f, r = _check(coords, feats, F_SMALL, np.eye(3), np.zeros(3), 1, (0.0, 0.0, 0.0), 1.0, 16)
    np.testing.assert_array_equal(r.cpu().numpy(), np.arange(len(coords)))
    np.testing.assert_allclose(f.cpu().numpy(), feats, rtol=0, atol=1e-6)
    Ri = sh.cube_rotations()[7].astype(np.float64)
    ctr = np.full(3, 8.5)
    _check(coords, feats, F_SMALL, Ri, ctr - Ri @ ctr, 1, (0.0, 0.0, 0.0), 1.0, 16)


def test_steer_rejects_non_rotations():
    coords = torch.zeros((1, 4), dtype=torch.int32, device=DEV)
    feats = torch.zeros((1, 1), device=DEV)
    for bad in (np.diag([1.0, 1.0, -1.0]), 2 * np.eye(3)):
        with pytest.raises(_abi.SSConvError) as e:
            P.steer(coords, feats, ((0, 1),), bad, np.zeros(3))
        assert e.value.code == _abi.E_INVALID

"""Pins for the oracle's Feature-Steering (Sec. 4.1).

* The identity motion returns the sparse tensor unchanged.
* Every 90-degree rotation of the cube group about a site centre, followed by a whole-voxel
  translation, maps site centres exactly onto site centres: the new sites equal the integer
  transform R (x - c) + c + t of the old ones (computed without floating point), and each new
  feature is the old one rotated by the block Wigner-D matrix.
* Steering commutes with the SS-Conv for those motions: conv(steer(F)) = steer(conv(F)) on a
  submanifold layer with fields of order 0, 1 and 2 (the equivariance that makes the module
  meaningful; it ties the Wigner-D convention to the steerable basis).
* A generic rotation merges sites; the count-weighted mean of the merged features conserves the
  sum of the rotated features, and |f| of every l = 1 field is preserved by the rotation alone.
"""
import numpy as np

from oracle import conv as oc
from oracle import rulebook as orb
from oracle import sh
from oracle import steer as ost
from workloads.configs import LayerSpec

FIELDS = ((0, 2), (1, 2), (2, 1))   # 2 + 6 + 5 = 13 channels


def _cloud(rng, n, grid, batch=2, margin=3):
    c = np.stack([rng.integers(0, batch, n)] + [rng.integers(margin, grid - margin, n) for _ in range(3)], 1)
    return np.unique(c, axis=0).astype(np.int32)


def test_identity_motion():
    rng = np.random.default_rng(1)
    c = _cloud(rng, 300, 16)
    f = rng.standard_normal((len(c), 13))
    c2, f2, row = ost.steer(c, f, FIELDS, np.eye(3), (0.0, 0.0, 0.0), (0.0, 0.0, 0.0), 1.0, 16)
    np.testing.assert_array_equal(c2, c)
    np.testing.assert_allclose(f2, f, rtol=0, atol=1e-12)
    np.testing.assert_array_equal(row, np.arange(len(c)))


def test_cube_rotations_map_sites_exactly():
    rng = np.random.default_rng(2)
    grid, vox, origin = 16, 0.5, np.array([-4.0, -4.0, -4.0])
    c = _cloud(rng, 200, grid)
    f = rng.standard_normal((len(c), 13))
    ctr = np.array([8, 8, 8])                         # a site; its centre is origin + 8.5 voxel
    p_ctr = origin + (ctr + 0.5) * vox
    for Ri in sh.cube_rotations():
        R = Ri.astype(np.float64)
        shift = np.array([1, -1, 2])
        t = p_ctr - R @ p_ctr + shift * vox              # rotate about the centre site, then shift
        c2, f2, row = ost.steer(c, f, FIELDS, R, t, origin, vox, grid)
        want_xyz = (c[:, 1:].astype(np.int64) - ctr) @ Ri.T + ctr + shift
        want = np.concatenate([c[:, :1].astype(np.int64), want_xyz], 1)
        order = np.lexsort(want.T[::-1])
        np.testing.assert_array_equal(c2, want[order].astype(np.int32))
        rho = sh.block_rep(FIELDS, R)
        np.testing.assert_allclose(f2, (f @ rho.T)[order], atol=1e-10)
        np.testing.assert_array_equal(row[order], np.arange(len(c)))


def test_steering_commutes_with_ssconv():
    rng = np.random.default_rng(3)
    grid = 16
    c = _cloud(rng, 250, grid, batch=1, margin=4)
    spec = LayerSpec(3, 1, True, FIELDS, ((0, 1), (1, 2), (2, 2)), shells=(0.0, 1.0))
    lay = oc.Layer(spec)
    kap = lay.kappa(rng.standard_normal(lay.n_coeff))
    f = rng.standard_normal((len(c), 13))
    out_fields = spec.fields_out

    def conv(coords, feats):
        R_ = orb.rulebook(coords, coords, 3, 1)
        return oc.forward(feats, R_, kap, len(coords))

    ctr, vox, origin = np.array([8, 8, 8]), 1.0, np.zeros(3)
    p_ctr = origin + (ctr + 0.5) * vox
    for Ri in sh.cube_rotations()[::5]:
        R = Ri.astype(np.float64)
        t = p_ctr - R @ p_ctr
        c_s, f_s, _ = ost.steer(c, f, FIELDS, R, t, origin, vox, grid)
        lhs = conv(c_s, f_s)
        c_o, rhs, _ = ost.steer(c, conv(c, f), out_fields, R, t, origin, vox, grid)
        np.testing.assert_array_equal(c_o, c_s)
        np.testing.assert_allclose(lhs, rhs, atol=1e-9)


def test_generic_rotation_merges_and_conserves():
    rng = np.random.default_rng(4)
    c = _cloud(rng, 400, 24, batch=1, margin=6)
    f = rng.standard_normal((len(c), 13))
    R = sh.axis_rotation(2, np.pi / 4) @ sh.axis_rotation(0, 0.3)
    origin, vox = np.zeros(3), 1.0
    ctr = np.full(3, 12.0)
    t = ctr - R @ ctr
    c2, f2, row = ost.steer(c, f, FIELDS, R, t, origin, vox, 24)
    assert len(c2) < len(c) and (row >= 0).all()
    counts = np.bincount(row, minlength=len(c2))
    rotated = f @ sh.block_rep(FIELDS, R).T
    np.testing.assert_allclose((counts[:, None] * f2).sum(0), rotated.sum(0), atol=1e-9)
    # rotation alone preserves the norm of every l = 1 field of every site
    for k in range(2):
        sl = slice(2 + 3 * k, 5 + 3 * k)
        np.testing.assert_allclose(np.linalg.norm(rotated[:, sl], axis=1), np.linalg.norm(f[:, sl], axis=1),
                                   rtol=1e-12)

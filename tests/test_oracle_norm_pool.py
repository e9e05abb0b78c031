"""Pins for the oracle's steerable normalisation (Sec. 3.3, Eq. 11) and sparse average pooling
(footnote of Sec. 3.1).

Norm: the normalised scalar channels have mean 0 and variance Var/(Var+eps), the normalised
l > 0 fields have E|y|^2 = nu/(nu+eps); with eps = 0 the result is invariant to scaling each
field and to shifting scalar channels; Norm commutes with rotating every field by its Wigner-D
matrix and with permuting the sites; the backward pass matches central finite differences.
Pooling: the output set equals a brute-force scan of the coarse grid; the values equal
torch's dense avg_pool3d of the zero-filled grid at active outputs (and that dense result
vanishes elsewhere); the backward pass is the exact adjoint; pooling commutes with the 24 cube
rotations about the grid centre and with even shifts.
"""
import numpy as np
import pytest

from oracle import norm_pool as npl
from oracle import sh

FIELDS = ((0, 3), (1, 2), (2, 1))   # 3 + 6 + 5 = 14 channels
C = 14


def _feats(n, seed):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((n, C)) * rng.uniform(0.5, 3.0, C) + rng.uniform(-2, 2, C)
    return x


def test_norm_statistics_closed_form():
    x = _feats(500, 0)
    y = npl.norm_forward(x, FIELDS)
    for l, c, d in npl._field_slices(FIELDS):
        f, g = x[:, c:c + d], y[:, c:c + d]
        if l == 0:
            assert abs(g.mean()) < 1e-12
            assert abs(g.var() - f.var() / (f.var() + npl.EPS)) < 1e-12
        else:
            nu = (f * f).sum(1).mean()
            assert abs((g * g).sum(1).mean() - nu / (nu + npl.EPS)) < 1e-12
            # l > 0 fields are only rescaled: no mean is subtracted
            ratio = g / f
            assert np.allclose(ratio, ratio[0, 0], rtol=1e-12)


def test_norm_scale_and_shift_invariance():
    x = _feats(300, 1)
    y = npl.norm_forward(x, FIELDS, eps=0.0)
    rng = np.random.default_rng(2)
    x2 = x.copy()
    for l, c, d in npl._field_slices(FIELDS):
        x2[:, c:c + d] *= rng.uniform(0.2, 5.0)
        if l == 0:
            x2[:, c] += rng.uniform(-3, 3)
    assert np.abs(npl.norm_forward(x2, FIELDS, eps=0.0) - y).max() < 1e-12


def test_norm_equivariance_and_site_permutation():
    x = _feats(200, 3)
    y = npl.norm_forward(x, FIELDS)
    perm = np.random.default_rng(4).permutation(len(x))
    for Rm in sh.cube_rotations()[::5] + [sh.axis_rotation(0, 0.7) @ sh.axis_rotation(2, -1.1)]:
        rho = sh.block_rep(FIELDS, Rm)
        ry = npl.norm_forward((x @ rho.T)[perm], FIELDS)
        assert np.abs(ry - (y @ rho.T)[perm]).max() < 1e-10


def test_norm_backward_finite_differences():
    x = _feats(40, 5)
    rng = np.random.default_rng(6)
    dy = rng.standard_normal(x.shape)
    dx = npl.norm_backward(x, dy, FIELDS)
    for t in range(4):
        d = rng.standard_normal(x.shape)
        h = 1e-6
        fd = ((npl.norm_forward(x + h * d, FIELDS) - npl.norm_forward(x - h * d, FIELDS)) * dy).sum() / (2 * h)
        assert abs(fd - (dx * d).sum()) < 1e-6 * max(1.0, abs(fd))
    # scalar channels: the gradient is orthogonal to constant shifts
    for l, c, _ in npl._field_slices(FIELDS):
        if l == 0:
            assert abs(dx[:, c].sum()) < 1e-10


def _coords(seed, n, grid, batch=1):
    rng = np.random.default_rng(seed)
    c = np.concatenate([rng.integers(0, batch, (n, 1)), rng.integers(0, grid, (n, 3))], 1)
    return np.unique(c, axis=0).astype(np.int32)


def test_pool_sites_bruteforce():
    grid = 8
    c = _coords(7, 120, grid, batch=2)
    got = npl.pool_sites(c)
    S = {tuple(v) for v in c.tolist()}
    want = []
    for b in range(2):
        for X in range(grid // 2):
            for Y in range(grid // 2):
                for Z in range(grid // 2):
                    if any((b, 2 * X + i, 2 * Y + j, 2 * Z + k) in S
                           for i in (0, 1) for j in (0, 1) for k in (0, 1)):
                        want.append((b, X, Y, Z))
    assert got.tolist() == [list(w) for w in want]


def test_pool_matches_dense_avg_pool3d():
    torch = pytest.importorskip("torch")
    grid, batch = 10, 2
    c = _coords(8, 300, grid, batch)
    x = np.random.default_rng(9).standard_normal((len(c), C))
    oc = npl.pool_sites(c)
    y = npl.pool_forward(x, npl.pool_members(c, oc), len(oc))
    dense = np.zeros((batch, C, grid, grid, grid))
    dense[c[:, 0], :, c[:, 1], c[:, 2], c[:, 3]] = x
    ref = torch.nn.functional.avg_pool3d(torch.from_numpy(dense), 2, 2).numpy()   # [B, C, G/2, ...]
    assert np.abs(ref[oc[:, 0], :, oc[:, 1], oc[:, 2], oc[:, 3]] - y).max() < 1e-13
    mask = np.ones(ref.shape[:1] + ref.shape[2:], bool)
    mask[oc[:, 0], oc[:, 1], oc[:, 2], oc[:, 3]] = False
    assert np.abs(ref.transpose(0, 2, 3, 4, 1)[mask]).max() == 0.0
    # the oracle's own dense reference agrees with torch's
    d2 = npl.dense_avg_pool(c, x, grid, batch)
    assert np.abs(d2 - ref.transpose(0, 2, 3, 4, 1)).max() < 1e-13


def test_pool_adjoint():
    c = _coords(10, 400, 12, batch=3)
    oc = npl.pool_sites(c)
    m = npl.pool_members(c, oc)
    rng = np.random.default_rng(11)
    x, g = rng.standard_normal((len(c), C)), rng.standard_normal((len(oc), C))
    lhs = (npl.pool_forward(x, m, len(oc)) * g).sum()
    rhs = (x * npl.pool_backward(g, m)).sum()
    assert abs(lhs - rhs) < 1e-12 * max(1.0, abs(lhs))


def test_pool_rotation_and_shift_equivariance():
    grid = 12
    c = _coords(12, 250, grid)
    x = np.random.default_rng(13).standard_normal((len(c), C))
    oc = npl.pool_sites(c)
    y = npl.pool_forward(x, npl.pool_members(c, oc), len(oc))
    ctr, octr = (grid - 1) / 2.0, (grid // 2 - 1) / 2.0     # windows map to windows about these
    for Rm in sh.cube_rotations():
        rc = c.copy()
        rc[:, 1:] = np.rint((c[:, 1:] - ctr) @ Rm.T + ctr).astype(np.int32)
        rho = sh.block_rep(FIELDS, Rm)
        roc = npl.pool_sites(rc)
        ry = npl.pool_forward(x @ rho.T, npl.pool_members(rc, roc), len(roc))
        want = oc.copy()
        want[:, 1:] = np.rint((oc[:, 1:] - octr) @ Rm.T + octr).astype(np.int32)
        where = {tuple(v): i for i, v in enumerate(roc.tolist())}
        perm = np.array([where[tuple(v)] for v in want.tolist()])
        assert np.abs(ry[perm] - y @ rho.T).max() < 1e-12
    sc = c.copy()
    sc[:, 1:] += np.array([2, 4, 0])
    soc = npl.pool_sites(sc)
    assert np.array_equal(soc[:, 1:], oc[:, 1:] + np.array([1, 2, 0]))
    assert np.abs(npl.pool_forward(x, npl.pool_members(sc, soc), len(soc)) - y).max() == 0.0

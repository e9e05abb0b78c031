"""Pins for the oracle's synthesis, forward, backward and gated nonlinearity.

(a) the sparse forward equals a brute-force dense convolution (Eq. 1 / Eq. 6)
    on the densified grid, and the dense result vanishes off the dilated set;
(b) exact equivariance under the 24 cube rotations (Eq. 2-4), features
    transformed by the Wigner-D matrix of each field;
(c) equivariance under integer shifts;
plus special cases (1x1x1 kernel = per-site GEMM, isolated site, isotropic
scalar kernel), the adjoint identity for the backward pass, exact linearity in
the coefficients and finite differences through the gate.
"""
import numpy as np
import pytest

from oracle import basis, conv, sh
from oracle import rulebook as rb
from workloads import CONFIGS
from workloads.configs import LayerSpec, gate_fields
from workloads.gen import make_coords, ellipsoid_dense, voxelise


def _layer_data(spec, coords, seed=0, grid=None):
    lay = conv.Layer(spec)
    rng = np.random.default_rng(seed)
    w = rng.standard_normal(lay.n_coeff)
    f = rng.standard_normal((len(coords), spec.cin))
    return lay, w, f


def _run(spec, lay, w, coords, feats, grid):
    out_c = rb.output_sites(coords, grid, spec.ksize, spec.stride, spec.submanifold)
    R = rb.rulebook(coords, out_c, spec.ksize, spec.stride)
    kap = lay.kappa(w)
    return out_c, R, kap, conv.forward(feats, R, kap, len(out_c))


def _sphere(radius, grid, centre=None, seed=0):
    rng = np.random.default_rng(seed)
    pts, _ = ellipsoid_dense(rng, np.full(3, radius))
    c = voxelise(pts + (np.full(3, grid / 2.0) if centre is None else centre), grid)
    return np.concatenate([np.zeros((len(c), 1), np.int64), c], 1).astype(np.int32)


MIXED = LayerSpec(5, 1, True, ((0, 2), (1, 2), (2, 1)), ((0, 1), (1, 1), (2, 2)), shells=(0.0, 1.0, 2.0))
MIXED3 = LayerSpec(3, 1, True, ((0, 2), (1, 1), (2, 1)), ((0, 2), (1, 2), (2, 1)), shells=(0.0, 1.0))
STRIDED = LayerSpec(3, 2, False, ((0, 2), (1, 1), (2, 1)), ((0, 1), (1, 2), (2, 1)), shells=(0.0, 1.0))
DILATE = LayerSpec(3, 1, False, ((0, 1), (1, 1)), ((0, 1), (1, 1)), shells=(0.0, 1.0))


def test_forward_loop_equals_vectorised():
    spec = CONFIGS[1].layers[0]
    c = make_coords(CONFIGS[1])
    lay, w, f = _layer_data(spec, c)
    out_c, R, kap, out = _run(spec, lay, w, c, f, 16)
    assert np.abs(out - conv.forward_loop(f, R, kap, len(out_c))).max() < 1e-12
    nbr = rb.neighbour_map(R, len(out_c))
    rows = np.arange(0, len(out_c), 7)
    assert np.abs(conv.forward_rows(f, nbr, kap, rows) - out[rows]).max() < 1e-12


@pytest.mark.parametrize("spec,grid,batch", [
    (CONFIGS[1].layers[0], 16, 1), (MIXED, 12, 1), (STRIDED, 12, 2), (DILATE, 10, 2)])
def test_forward_matches_dense_convolution(spec, grid, batch):
    if spec is CONFIGS[1].layers[0]:
        c = make_coords(CONFIGS[1])
    else:
        rng = np.random.default_rng(grid)
        c = np.concatenate([rng.integers(0, batch, (70, 1)), rng.integers(0, grid, (70, 3))], 1)
        c = np.unique(c, axis=0).astype(np.int32)
    lay, w, f = _layer_data(spec, c, seed=grid)
    out_c, R, kap, out = _run(spec, lay, w, c, f, grid)
    dense = conv.dense_conv(c, f, kap, grid, spec.stride, batch)
    got = dense[out_c[:, 0], out_c[:, 1], out_c[:, 2], out_c[:, 3]]
    assert np.abs(got - out).max() < 1e-12 * max(1.0, np.abs(out).max())
    if not spec.submanifold:                               # off the dilated set the dense result is exactly 0
        mask = np.ones(dense.shape[:4], bool)
        mask[out_c[:, 0], out_c[:, 1], out_c[:, 2], out_c[:, 3]] = False
        assert np.abs(dense[mask]).max() == 0.0


def test_forward_matches_torch_conv3d():
    """A library convolution (cross-correlation, so the kernel is flipped) agrees on the 16^3 workload."""
    torch = pytest.importorskip("torch")
    spec = CONFIGS[1].layers[0]
    c = make_coords(CONFIGS[1])
    lay, w, f = _layer_data(spec, c, seed=4)
    out_c, R, kap, out = _run(spec, lay, w, c, f, 16)
    x = np.zeros((1, spec.cin, 16, 16, 16))
    x[0][:, c[:, 1], c[:, 2], c[:, 3]] = f.T
    k = kap.reshape(3, 3, 3, spec.cout, spec.cin)[::-1, ::-1, ::-1].transpose(3, 4, 0, 1, 2).copy()
    y = torch.nn.functional.conv3d(torch.from_numpy(x), torch.from_numpy(k), padding=1).numpy()
    got = y[0][:, c[:, 1], c[:, 2], c[:, 3]].T
    assert np.abs(got - out).max() < 1e-12 * np.abs(out).max()


def _rotate_case(spec, coords, feats, w, lay, Rm, centre, grid):
    rc = coords.copy()
    rc[:, 1:] = np.rint((coords[:, 1:] - centre) @ Rm.T + centre).astype(np.int32)
    rf = feats @ sh.block_rep(spec.fields_in, Rm).T
    return rc, rf


@pytest.mark.parametrize("which", ["c1", "mixed5", "mixed3"])
def test_rotation_equivariance_submanifold(which):
    if which == "c1":
        spec, grid = CONFIGS[1].layers[0], 16
        c = make_coords(CONFIGS[1])
    else:
        spec, grid = (MIXED, 12) if which == "mixed5" else (MIXED3, 12)
        c = _sphere(3.5, grid)
    lay, w, f = _layer_data(spec, c, seed=2)
    _, _, _, out = _run(spec, lay, w, c, f, grid)
    centre = (grid - 1) / 2.0
    worst = 0.0
    for Rm in sh.cube_rotations():
        rc, rf = _rotate_case(spec, c, f, w, lay, Rm, centre, grid)
        _, _, _, rout = _run(spec, lay, w, rc, rf, grid)      # submanifold: rows keep their order
        worst = max(worst, np.abs(rout - out @ sh.block_rep(spec.fields_out, Rm).T).max())
    assert worst < 1e-10 * max(1.0, np.abs(out).max())


def test_rotation_equivariance_stride2():
    spec, grid = STRIDED, 16
    c = _sphere(4.0, grid, centre=np.array([8.3, 7.6, 8.1]))
    lay, w, f = _layer_data(spec, c, seed=3)
    out_c, _, _, out = _run(spec, lay, w, c, f, grid)
    centre = 8.0                                           # even lattice point: outputs rotate about 4
    for Rm in sh.cube_rotations():
        rc, rf = _rotate_case(spec, c, f, w, lay, Rm, centre, grid)
        rout_c, _, _, rout = _run(spec, lay, w, rc, rf, grid)
        want_c = out_c.copy()
        want_c[:, 1:] = np.rint((out_c[:, 1:] - centre / 2) @ Rm.T + centre / 2).astype(np.int32)
        where = {tuple(x): i for i, x in enumerate(rout_c.tolist())}
        assert len(where) == len(want_c)
        perm = np.array([where[tuple(x)] for x in want_c.tolist()])
        err = np.abs(rout[perm] - out @ sh.block_rep(spec.fields_out, Rm).T).max()
        assert err < 1e-10 * np.abs(out).max()


def test_translation_equivariance():
    for spec, t in ((MIXED3, np.array([1, -2, 3])), (STRIDED, np.array([2, 4, -2]))):
        c = _sphere(3.0, 14, centre=np.array([7.2, 7.9, 6.6]))
        lay, w, f = _layer_data(spec, c, seed=5)
        out_c, _, _, out = _run(spec, lay, w, c, f, 20)
        cs = c.copy()
        cs[:, 1:] += t
        sout_c, _, _, sout = _run(spec, lay, w, cs, f, 20)
        assert np.array_equal(sout_c[:, 1:], out_c[:, 1:] + t // spec.stride)
        assert np.abs(sout - out).max() < 1e-12 * np.abs(out).max()


def test_special_cases():
    # 1x1x1 kernel: a per-site GEMM with kappa(0)
    spec = LayerSpec(1, 1, True, ((0, 3), (1, 1)), ((0, 2), (1, 2)), shells=(0.0,))
    c = _sphere(3.0, 10)
    lay, w, f = _layer_data(spec, c, seed=6)
    _, _, kap, out = _run(spec, lay, w, c, f, 10)
    assert np.abs(out - f @ kap[0].T).max() < 1e-13
    # an isolated site only sees kappa(0)
    spec = MIXED3
    c1 = np.array([[0, 5, 5, 5]], np.int32)
    lay, w, f = _layer_data(spec, c1, seed=7)
    _, _, kap, out = _run(spec, lay, w, c1, f, 10)
    assert np.abs(out[0] - kap[13] @ f[0]).max() < 1e-13
    # all-scalar fields: kappa(s) depends on |s| only (a radially symmetric stencil)
    spec = LayerSpec(3, 1, True, ((0, 2),), ((0, 3),), shells=(0.0, 1.0))
    lay = conv.Layer(spec)
    kap = lay.kappa(np.random.default_rng(8).standard_normal(lay.n_coeff))
    r2 = (basis.offsets(3) ** 2).sum(1)
    for v in np.unique(r2):
        same = kap[r2 == v]
        assert np.abs(same - same[0]).max() < 1e-15


def test_backward_adjoint_and_coeff_linearity():
    for spec, grid, batch in ((MIXED, 12, 1), (STRIDED, 12, 2)):
        rng = np.random.default_rng(11)
        c = np.concatenate([rng.integers(0, batch, (90, 1)), rng.integers(0, grid, (90, 3))], 1)
        c = np.unique(c, axis=0).astype(np.int32)
        lay, w, f = _layer_data(spec, c, seed=12)
        out_c, R, kap, out = _run(spec, lay, w, c, f, grid)
        g = rng.standard_normal(out.shape)
        d_in, dk = conv.backward(f, g, R, kap, len(c))
        # <conv(x), g> = <x, conv^T(g)>
        assert abs((out * g).sum() - (f * d_in).sum()) < 1e-11 * abs((out * g).sum())
        # L = <out, g> is linear in w: L(w + d) - L(w) = <dcoeff, d>
        dw = conv.synth_adjoint(spec, lay.basis, dk)
        d = rng.standard_normal(lay.n_coeff)
        out2 = conv.forward(f, R, lay.kappa(w + d), len(out_c))
        assert abs(((out2 - out) * g).sum() - dw @ d) < 1e-10 * max(1.0, abs(dw @ d))
        # loop form of dkappa
        dk_loop = np.zeros_like(dk)
        for si, r in enumerate(R):
            for o, i in r:
                dk_loop[si] += np.outer(g[o], f[i])
        assert np.abs(dk - dk_loop).max() < 1e-12


def test_gate_finite_differences():
    fields = ((0, 2), (1, 2), (2, 1))
    C = sum(m * (2 * l + 1) for l, m in fields)
    ng = 3
    rng = np.random.default_rng(13)
    x = rng.standard_normal((5, C + ng))
    x[np.abs(x) < 1e-3] = 0.5                                  # keep away from the ReLU kink
    dy = rng.standard_normal((5, C))
    dx = conv.gate_backward(x, dy, fields)
    h = 1e-6
    num = np.zeros_like(x)
    for idx in np.ndindex(*x.shape):
        xp, xm = x.copy(), x.copy()
        xp[idx] += h
        xm[idx] -= h
        num[idx] = ((conv.gate_forward(xp, fields) - conv.gate_forward(xm, fields)) * dy).sum() / (2 * h)
    assert np.abs(num - dx).max() < 1e-7
    # forward: ReLU on scalars, sigmoid(gate) * f on the others
    y = conv.gate_forward(x, fields)
    assert np.allclose(y[:, :2], np.maximum(x[:, :2], 0))
    assert np.allclose(y[:, 2:5], x[:, 2:5] / (1 + np.exp(-x[:, C:C + 1])))
    assert np.allclose(y[:, 8:13], x[:, 8:13] / (1 + np.exp(-x[:, C + 2:C + 3])))


def test_gated_stack_rotation_equivariance():
    """Two gated layers (submanifold then stride 2): scalar gates keep the stack equivariant."""
    F1 = ((0, 2), (1, 1), (2, 1))
    L1 = LayerSpec(3, 1, True, ((0, 2),), gate_fields(F1), shells=(0.0, 1.0), gated=True)
    L2 = LayerSpec(3, 2, False, F1, ((0, 1), (1, 1)), shells=(0.0, 1.0))
    grid = 16
    c = _sphere(4.0, grid, centre=np.array([8.4, 7.7, 8.2]))
    lays = [conv.Layer(L1), conv.Layer(L2)]
    rng = np.random.default_rng(14)
    ws = [rng.standard_normal(l.n_coeff) for l in lays]
    f0 = rng.standard_normal((len(c), 2))

    def stack(coords, f):
        o1, R1, k1, y1 = _run(L1, lays[0], ws[0], coords, f, grid)
        h = conv.gate_forward(y1, F1)
        return _run(L2, lays[1], ws[1], o1, h, grid)

    out_c, _, _, out = stack(c, f0)
    for Rm in sh.cube_rotations()[1::4]:
        rc = c.copy()
        rc[:, 1:] = np.rint((c[:, 1:] - 8.0) @ Rm.T + 8.0).astype(np.int32)
        rout_c, _, _, rout = stack(rc, f0)                     # scalar inputs: rho_in = identity
        want_c = out_c.copy()
        want_c[:, 1:] = np.rint((out_c[:, 1:] - 4.0) @ Rm.T + 4.0).astype(np.int32)
        where = {tuple(x): i for i, x in enumerate(rout_c.tolist())}
        perm = np.array([where[tuple(x)] for x in want_c.tolist()])
        err = np.abs(rout[perm] - out @ sh.block_rep(L2.fields_out, Rm).T).max()
        assert err < 1e-10 * np.abs(out).max()

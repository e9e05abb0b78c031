"""Pins for the oracle's spherical harmonics, Wigner-D matrices and steerable basis.

Every check here compares the oracle with something other than itself:
quadrature, closed forms, group axioms, the selection rule behind Eq. 7, the
kernel constraint of Eq. 4 evaluated exactly on the cube group, Schur's lemma
at the origin and the parameter count printed in Sec. 3.2.1.
"""
import json
import os
from math import pi, sqrt

import numpy as np
import pytest

from oracle import basis, sh
from oracle.conv import synth, Layer
from workloads import CONFIGS
from workloads.configs import LayerSpec

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _quadrature(n_t=10, n_p=21):
    x, w = np.polynomial.legendre.leggauss(n_t)          # exact in cos(theta) to degree 2 n_t - 1
    ph = np.arange(n_p) * 2 * pi / n_p                    # exact for trig degree < n_p
    ct, pp = np.meshgrid(x, ph, indexing="ij")
    st = np.sqrt(1 - ct ** 2)
    dirs = np.stack([st * np.cos(pp), st * np.sin(pp), ct], -1).reshape(-1, 3)
    wt = (w[:, None] * np.full(n_p, 2 * pi / n_p)[None]).reshape(-1)
    return dirs, wt


@pytest.mark.parametrize("J1", range(5))
@pytest.mark.parametrize("J2", range(5))
def test_sh_orthonormal(J1, J2):
    dirs, wt = _quadrature()
    G = (sh.real_sh(J1, dirs) * wt[:, None]).T @ sh.real_sh(J2, dirs)
    ref = np.eye(2 * J1 + 1) if J1 == J2 else np.zeros_like(G)
    assert np.abs(G - ref).max() < 1e-13


def test_sh_l1_closed_form_golden():
    g = json.load(open(os.path.join(GOLDEN, "real_sh_l1.json")))
    pts = np.array(g["points"], float)
    want = np.array(g["values_over_sqrt_3_over_4pi"], float) * sqrt(3 / (4 * pi))
    assert np.abs(sh.real_sh(1, pts) - want).max() < 1e-15


def test_sh_l2_closed_form():
    # independent closed forms of the real l=2 harmonics (no Condon-Shortley phase)
    u = sh.random_dirs(50, seed=3)
    x, y, z = u.T
    c = sqrt(15 / (4 * pi))
    want = np.stack([c * x * y, c * y * z, sqrt(5 / (16 * pi)) * (3 * z * z - 1), c * x * z,
                     0.5 * c * (x * x - y * y)], 1)
    assert np.abs(sh.real_sh(2, u) - want).max() < 1e-14


def test_sh_origin_reading():
    z = np.zeros((1, 3))
    assert abs(sh.real_sh(0, z)[0, 0] - 1 / (2 * sqrt(pi))) < 1e-15
    for J in range(1, 5):
        assert np.all(sh.real_sh(J, z) == 0)


@pytest.mark.parametrize("J", range(5))
def test_wigner_d_properties(J):
    rng = np.random.default_rng(J)
    from workloads.gen import random_rotation
    R1, R2 = random_rotation(rng), random_rotation(rng)
    D1, D2, D12 = sh.wigner_d(J, R1), sh.wigner_d(J, R2), sh.wigner_d(J, R1 @ R2)
    assert sh.wigner_d_residual(J, R1, D1) < 1e-12
    assert np.abs(D1 @ D1.T - np.eye(2 * J + 1)).max() < 1e-12
    assert np.abs(D12 - D1 @ D2).max() < 1e-12


def test_wigner_d1_is_permuted_rotation():
    from workloads.gen import random_rotation
    R = random_rotation(np.random.default_rng(5))
    P = np.zeros((3, 3))
    P[0, 1] = P[1, 2] = P[2, 0] = 1.0                      # (x, y, z) -> (y, z, x)
    assert np.abs(sh.wigner_d(1, R) - P @ R @ P.T).max() < 1e-12


@pytest.mark.parametrize("J", range(5))
def test_wigner_d_quarter_turn_order_four(J):
    R = sh.axis_rotation(2, pi / 2)
    D = sh.wigner_d(J, R)
    assert np.abs(np.linalg.matrix_power(D, 4) - np.eye(2 * J + 1)).max() < 1e-12


def test_cube_group():
    rots = sh.cube_rotations()
    assert len(rots) == 24
    keys = {tuple(r.reshape(-1)) for r in rots}
    for a in rots:
        for b in rots:
            assert tuple((a @ b).reshape(-1)) in keys


@pytest.mark.parametrize("k", range(3))
@pytest.mark.parametrize("l", range(3))
def test_selection_rule_and_gap(k, l):
    """The constraint has a 1-dim solution iff |k-l| <= J <= k+l (the range of Eq. 7), else none."""
    for J in range(6):
        sv, _ = basis.constraint_singular_values(k, l, J)
        null = int((sv < 1e-8).sum())
        assert null == (1 if abs(k - l) <= J <= k + l else 0)
        nxt = sv[null] if null < len(sv) else np.inf
        assert nxt > 1e-2                                   # clear spectral gap


def test_intertwiner_special_forms():
    for k in range(3):
        Q = basis.intertwiner(k, k, 0)[0]
        assert np.abs(Q / Q[0, 0] - np.eye(2 * k + 1)).max() < 1e-12
    Q = basis.intertwiner(1, 1, 1)
    eps = np.zeros((3, 3, 3))
    for (a, b, c), sgn in {(0, 1, 2): 1, (1, 2, 0): 1, (2, 0, 1): 1, (0, 2, 1): -1, (2, 1, 0): -1, (1, 0, 2): -1}.items():
        eps[a, b, c] = sgn
    ratio = Q[0, 1, 2] / eps[0, 1, 2]
    assert np.abs(Q - ratio * eps).max() < 1e-12


@pytest.mark.parametrize("ksize,shells", [(3, (0.0, 1.0)), (5, (0.0, 1.0, 2.0)), (3, (0.0, 1.0, sqrt(2), sqrt(3)))])
def test_basis_exactly_steerable_on_cube_group(ksize, shells):
    """Eq. 4: B(R s) = D^k(R) B(s) D^l(R)^T for all 24 rotations that map the grid S to itself."""
    S = basis.offsets(ksize)
    worst = 0.0
    for k in range(3):
        for l in range(3):
            B = basis.pair_basis(k, l, shells, 0.6, ksize, None)
            for R in sh.cube_rotations():
                idx = [basis.offset_index(ksize, R @ s) for s in S]
                rhs = np.einsum("ab,qsbc,dc->qsad", sh.wigner_d(k, R), B, sh.wigner_d(l, R))
                worst = max(worst, np.abs(B[:, idx] - rhs).max())
    assert worst < 1e-13


def test_basis_schur_at_origin():
    """kappa(0) commutes with every rotation: nonzero only for k = l, J = 0, and then a multiple of I."""
    ksize = 3
    o = basis.offset_index(ksize, (0, 0, 0))
    for k in range(3):
        for l in range(3):
            for J in basis.j_range(k, l, None):
                B0 = basis.raw_basis_kernel(k, l, J, 0.0, 0.6, ksize)[o]
                if k == l and J == 0:
                    assert np.abs(B0 / B0[0, 0] - np.eye(2 * k + 1)).max() < 1e-12
                else:
                    assert np.abs(B0).max() < 1e-15


def test_basis_normalisation():
    B = basis.pair_basis(2, 1, (0.0, 1.0), 0.6, 3, None)
    assert np.allclose((B ** 2).sum((1, 2, 3)), 1.0, atol=1e-14)
    for q in range(B.shape[0]):
        f = B[q].reshape(-1)
        first = f[np.argmax(np.abs(f) > 1e-3 * np.abs(f).max())]
        assert first > 0


def test_param_counts_golden():
    """Sec. 3.2.1: M [2 min(k,l) + 1] learnable scalars per block (J uncapped)."""
    g = json.load(open(os.path.join(GOLDEN, "param_counts.json")))
    for b in g["blocks"]:
        spec = LayerSpec(3, 1, True, ((b["l"], 1),), ((b["k"], 1),), shells=tuple(range(b["M"])))
        assert basis.coeff_count(spec) == b["count"] == basis.paper_param_count(b["k"], b["l"], b["M"])


def test_workload_coeff_counts():
    want = {1: [64], 2: [7488], 3: [4416], 4: [23040], 5: [1536, 23040, 30720, 30720, 23040]}
    for i, counts in want.items():
        assert [basis.coeff_count(L) for L in CONFIGS[i].layers] == counts


def test_synth_one_hot_reproduces_basis_element():
    """Eq. 7 is linear in w: a one-hot w yields exactly one normalised basis element in one block."""
    from oracle.conv import coeff_blocks
    spec = LayerSpec(3, 1, True, ((0, 1), (1, 2)), ((1, 1), (2, 1)), shells=(0.0, 1.0))
    lay = Layer(spec)
    blocks = list(coeff_blocks(spec, lay.basis))
    for q in np.random.default_rng(0).choice(lay.n_coeff, 8, replace=False):
        w = np.zeros(lay.n_coeff)
        w[q] = 1.0
        kap = synth(spec, lay.basis, w)
        ro, k, ci, l, off, nq = next(b for b in blocks if b[4] <= q < b[4] + b[5])
        want = np.zeros_like(kap)
        want[:, ro:ro + 2 * k + 1, ci:ci + 2 * l + 1] = lay.basis[(k, l)][q - off]
        assert np.abs(kap - want).max() == 0.0

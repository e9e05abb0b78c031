"""Pins for the oracle's output site sets and rule books.

The dict-based rule book is checked against the literal all-pairs loop of
Alg. 1, the dilated output set against Eq. 10 evaluated at every grid site,
and both against the symmetries the definitions imply (submanifold identity
offset, R_s / R_-s symmetry, rotation and shift covariance).
"""
import numpy as np
import pytest

from oracle import basis, sh
from oracle import rulebook as rb
from workloads import CONFIGS
from workloads.gen import make_coords


def _random_sites(seed, n, grid, batch=1):
    rng = np.random.default_rng(seed)
    c = np.concatenate([rng.integers(0, batch, (n, 1)), rng.integers(0, grid, (n, 3))], 1)
    return np.unique(c, axis=0).astype(np.int32)


def _same(a, b):
    return rb.pair_set(a) == rb.pair_set(b)


def test_c1_rulebook_matches_algorithm1_loop():
    spec = CONFIGS[1]
    c = make_coords(spec)
    R = rb.rulebook(c, c, 3, 1)
    assert _same(R, rb.rulebook_bruteforce(c, c, 3, 1))
    assert sum(len(r) for r in R) > 5 * len(c)


@pytest.mark.parametrize("ksize,stride,batch", [(3, 1, 1), (5, 1, 2), (3, 2, 2), (5, 2, 1)])
def test_random_rulebooks_match_algorithm1(ksize, stride, batch):
    c = _random_sites(ksize * 10 + stride, 60, 9, batch)
    out = rb.output_sites(c, 9, ksize, stride, submanifold=False)
    assert _same(rb.rulebook(c, out, ksize, stride), rb.rulebook_bruteforce(c, out, ksize, stride))
    if stride == 1:
        assert _same(rb.rulebook(c, c, ksize, 1), rb.rulebook_bruteforce(c, c, ksize, 1))


@pytest.mark.parametrize("ksize,stride", [(3, 1), (3, 2), (5, 2), (5, 1)])
def test_output_sites_match_eq10(ksize, stride):
    c = _random_sites(7 + ksize + stride, 40, 8, batch=2)
    got = rb.output_sites(c, 8, ksize, stride, submanifold=False)
    want = rb.output_sites_bruteforce(c, 8, ksize, stride)
    assert np.array_equal(got, want)                     # same set, same lexicographic order


def test_stride2_grid_shape():
    c = np.array([[0, 0, 0, 0], [0, 63, 63, 63]], np.int32)
    out = rb.output_sites(c, 64, 3, 2, submanifold=False)
    assert out[:, 1:].min() == 0 and out[:, 1:].max() == 31


def test_submanifold_identity_offset_and_symmetry():
    c = make_coords(CONFIGS[1])
    R = rb.rulebook(c, c, 3, 1)
    centre = basis.offset_index(3, (0, 0, 0))
    assert np.array_equal(R[centre], np.stack([np.arange(len(c))] * 2, 1))
    S = basis.offsets(3)
    for si, s in enumerate(S):
        mirror = R[basis.offset_index(3, -s)]
        assert {tuple(p) for p in R[si].tolist()} == {(i, o) for o, i in mirror.tolist()}


def test_rulebook_rotation_covariance():
    """Rotating the sites by a cube rotation about the grid centre maps R_s to R_{R s}."""
    c = make_coords(CONFIGS[1])
    G = CONFIGS[1].grid
    R0 = rb.rulebook(c, c, 3, 1)
    S = basis.offsets(3)
    ctr = (G - 1) / 2.0
    for Rm in sh.cube_rotations()[::5]:
        rc = c.copy()
        rc[:, 1:] = np.rint((c[:, 1:] - ctr) @ Rm.T + ctr).astype(np.int32)
        R1 = rb.rulebook(rc, rc, 3, 1)
        for si, s in enumerate(S):
            assert rb.pair_set([R0[si]]) == rb.pair_set([R1[basis.offset_index(3, Rm @ s)]])


def test_rulebook_shift_covariance():
    c = _random_sites(3, 80, 8, batch=2)                  # away from the far edge of a 10^3 grid
    out = rb.output_sites(c, 10, 3, 2, False)
    R0 = rb.rulebook(c, out, 3, 2)
    t = np.array([2, 4, 6])                                # even shift moves outputs by t/2
    cs = c.copy()
    cs[:, 1:] += t
    outs = rb.output_sites(cs, 20, 3, 2, False)
    assert np.array_equal(outs[:, 1:], out[:, 1:] + t // 2)
    assert _same(R0, rb.rulebook(cs, outs, 3, 2))


def test_batches_never_pair():
    c = np.array([[0, 3, 3, 3], [1, 3, 3, 4]], np.int32)
    R = rb.rulebook(c, c, 3, 1)
    for r in R:
        for o, i in r:
            assert c[o, 0] == c[i, 0]


def test_duplicate_sites_rejected():
    c = np.array([[0, 1, 1, 1], [0, 1, 1, 1]], np.int32)
    with pytest.raises(ValueError):
        rb.rulebook(c, c, 3, 1)


def test_empty_input():
    c = np.zeros((0, 4), np.int32)
    out = rb.output_sites(c, 8, 3, 2, False)
    assert out.shape == (0, 4)
    assert all(len(r) == 0 for r in rb.rulebook(c, out, 3, 2))

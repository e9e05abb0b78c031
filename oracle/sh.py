"""Real spherical harmonics and Wigner-D matrices (oracle; test infrastructure only).

Sec. 3.1 (Eq. 5): a feature is a stack of irreducible fields, each of order l,
transforming by a (2l+1)x(2l+1) Wigner-D matrix.  Sec. 3.2.1 (Eq. 8) builds
kernels from spherical harmonics Y^J.  The paper fixes neither real/complex
form, normalisation nor phase; this oracle reads them as real, orthonormal on
the sphere, ordered j = -J..J, with no Condon-Shortley phase:

    Y_J^0       = N_J^0 P_J^0(cos t)
    Y_J^{j>0}   = sqrt2 N_J^j P_J^j(cos t) cos(j p)
    Y_J^{j<0}   = sqrt2 N_J^|j| P_J^|j|(cos t) sin(|j| p)
    N_J^j       = sqrt((2J+1)/(4 pi) (J-j)!/(J+j)!)

so that Y_1 = sqrt(3/(4 pi)) (y, z, x)/r.  The Wigner-D matrix of order J is
*defined* by Y^J(R u) = D^J(R) Y^J(u) and computed by least squares over
random directions, so it is exactly the representation the harmonics carry.
"""
from itertools import permutations, product
from math import factorial, pi, sqrt

import numpy as np
from scipy.special import lpmv


def real_sh(J: int, dirs: np.ndarray) -> np.ndarray:
    """Y^J at unit (or zero) vectors ``dirs`` [n,3] -> [n, 2J+1] (fp64).

    At the zero vector the direction is undefined; the oracle takes
    Y^0 = 1/(2 sqrt(pi)) and Y^{J>0} = 0 there (pinned by Schur's lemma on
    the kernel at the origin).
    """
    d = np.asarray(dirs, np.float64).reshape(-1, 3)
    r = np.linalg.norm(d, axis=1)
    zero = r < 1e-12
    u = np.where(zero[:, None], np.array([0.0, 0.0, 1.0]), d / np.where(zero, 1.0, r)[:, None])
    ct = np.clip(u[:, 2], -1.0, 1.0)
    ph = np.arctan2(u[:, 1], u[:, 0])
    out = np.zeros((len(d), 2 * J + 1))
    for j in range(-J, J + 1):
        m = abs(j)
        nrm = sqrt((2 * J + 1) / (4 * pi) * factorial(J - m) / factorial(J + m))
        p = (-1.0) ** m * lpmv(m, J, ct)  # scipy includes the Condon-Shortley phase; undo it
        if j == 0:
            val = nrm * p
        elif j > 0:
            val = sqrt(2.0) * nrm * p * np.cos(m * ph)
        else:
            val = sqrt(2.0) * nrm * p * np.sin(m * ph)
        out[:, j + J] = val
    if J > 0:
        out[zero] = 0.0
    return out


def random_dirs(n: int, seed: int = 0) -> np.ndarray:
    u = np.random.default_rng(seed).standard_normal((n, 3))
    return u / np.linalg.norm(u, axis=1, keepdims=True)


def wigner_d(J: int, R: np.ndarray, n_dirs: int = 96) -> np.ndarray:
    """D^J(R) with Y^J(R u) = D^J(R) Y^J(u), by least squares over random directions."""
    if J == 0:
        return np.ones((1, 1))
    u = random_dirs(n_dirs, seed=1000 + J)
    A = real_sh(J, u)
    B = real_sh(J, u @ np.asarray(R, np.float64).T)
    Dt, *_ = np.linalg.lstsq(A, B, rcond=None)
    return Dt.T


def wigner_d_residual(J: int, R: np.ndarray, D: np.ndarray, n_dirs: int = 200) -> float:
    u = random_dirs(n_dirs, seed=7)
    return float(np.abs(real_sh(J, u @ R.T) - real_sh(J, u) @ D.T).max())


def block_rep(fields, R) -> np.ndarray:
    """Block-diagonal representation rho(R) = (+) D^{l_i}(R) for a field list ((l, mult), ...)."""
    blocks = []
    cache = {}
    for l, mult in fields:
        if l not in cache:
            cache[l] = wigner_d(l, R)
        blocks += [cache[l]] * mult
    n = sum(b.shape[0] for b in blocks)
    out = np.zeros((n, n))
    o = 0
    for b in blocks:
        k = b.shape[0]
        out[o:o + k, o:o + k] = b
        o += k
    return out


def cube_rotations():
    """The 24 proper rotations of the cube: signed permutation matrices with det +1."""
    mats = []
    for perm in permutations(range(3)):
        for signs in product((-1, 1), repeat=3):
            M = np.zeros((3, 3), np.int64)
            for r, c in enumerate(perm):
                M[r, c] = signs[r]
            if round(np.linalg.det(M)) == 1:
                mats.append(M)
    return mats


def axis_rotation(axis: int, angle: float) -> np.ndarray:
    c, s = np.cos(angle), np.sin(angle)
    i, j = [a for a in range(3) if a != axis]
    R = np.eye(3)
    R[i, i], R[i, j], R[j, i], R[j, j] = c, -s, s, c
    return R

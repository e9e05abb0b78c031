"""Steerable basis kernels on the s^3 grid (oracle; test infrastructure only).

Sec. 3.2.1, Eq. 7-9.  For an output field of order k and an input field of
order l, the kernel is a linear combination of basis kernels

    kappa^{kl,Jm}(x) = phi^m(|x|) sum_j Y^J_j(x/|x|) Q^{kl,J}_j          (Eq. 8)
    phi^m(r)        = exp(-(r - m)^2 / (2 eps^2))

with J = |k-l| .. k+l (Eq. 7) and learned weights w^{kl,Jm}.  The paper writes
the change-of-basis matrix as Q^{kl}_j; the oracle reads it as Q^{kl,J}_j, the
(essentially unique) solution of the steerability constraint of Eq. 4 applied
to Eq. 8:

    sum_j D^J(R)_{j j'} Q_j = D^k(R) Q_{j'} D^l(R)^T   for all rotations R.

It is computed here as the SVD null space of that linear system stacked for
two generic rotations (no Clebsch-Gordan tables are used).

The paper leaves the basis normalisation open; each element (k,l,J,m) is
scaled to unit Frobenius norm over (offset, row, column) and its sign is
chosen so that the first entry (row-major over offset, row, column) whose
magnitude exceeds 1e-3 of the element's largest magnitude is positive.  This
removes every phase/scale convention from the comparison with an independent
builder.  An optional band limit ``jmax`` drops whole J blocks, which keeps
the kernel exactly steerable.
"""
from functools import lru_cache
from math import sqrt
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from .sh import real_sh, wigner_d

SIGN_REL_THRESHOLD = 1e-3


def offsets(ksize: int) -> np.ndarray:
    """Kernel offsets s in S = {-(s-1)/2 .. (s-1)/2}^3 (Sec. 3.2, Eq. 6) as [ksize^3, 3] int.

    Row index s_idx = ((dx+h)*ksize + (dy+h))*ksize + (dz+h), h = (ksize-1)/2.
    """
    h = (ksize - 1) // 2
    r = np.arange(-h, h + 1)
    g = np.stack(np.meshgrid(r, r, r, indexing="ij"), -1).reshape(-1, 3)
    return g.astype(np.int64)


def offset_index(ksize: int, s) -> int:
    h = (ksize - 1) // 2
    dx, dy, dz = (int(v) for v in s)
    return ((dx + h) * ksize + (dy + h)) * ksize + (dz + h)


def _random_rotations(n: int, seed: int) -> List[np.ndarray]:
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        q = rng.standard_normal(4)
        q /= np.linalg.norm(q)
        w, x, y, z = q
        out.append(np.array([
            [1 - 2 * (y * y + z * z), 2 * (x * y - z * w), 2 * (x * z + y * w)],
            [2 * (x * y + z * w), 1 - 2 * (x * x + z * z), 2 * (y * z - x * w)],
            [2 * (x * z - y * w), 2 * (y * z + x * w), 1 - 2 * (x * x + y * y)]]))
    return out


def constraint_singular_values(k: int, l: int, J: int, n_rot: int = 2, seed: int = 31):
    """Singular values (ascending) and right singular vectors of the stacked constraint."""
    dJ, dk, dl = 2 * J + 1, 2 * k + 1, 2 * l + 1
    blocks = []
    for R in _random_rotations(n_rot, seed):
        DJ, Dk, Dl = wigner_d(J, R), wigner_d(k, R), wigner_d(l, R)
        lhs = np.kron(DJ.T, np.eye(dk * dl))
        rhs = np.kron(np.eye(dJ), np.kron(Dk, Dl))
        blocks.append(lhs - rhs)
    A = np.vstack(blocks)
    _, sv, vt = np.linalg.svd(A)
    order = np.argsort(sv)
    return sv[order], vt[order]


@lru_cache(maxsize=None)
def intertwiner(k: int, l: int, J: int) -> Optional[np.ndarray]:
    """Q^{kl,J} as [2J+1, 2k+1, 2l+1], or None when the solution space is empty."""
    sv, vt = constraint_singular_values(k, l, J)
    null = sv < 1e-8
    if not null.any():
        return None
    assert null.sum() == 1, (k, l, J, sv[:3])
    return vt[0].reshape(2 * J + 1, 2 * k + 1, 2 * l + 1)


def radial(r: np.ndarray, m: float, eps: float) -> np.ndarray:
    """Gaussian radial profile phi^m(r) of Eq. 8."""
    return np.exp(-0.5 * (r - m) ** 2 / eps ** 2)


def raw_basis_kernel(k: int, l: int, J: int, m: float, eps: float, ksize: int) -> Optional[np.ndarray]:
    """Eq. 8 on the grid before normalisation: [ksize^3, 2k+1, 2l+1]."""
    Q = intertwiner(k, l, J)
    if Q is None:
        return None
    S = offsets(ksize).astype(np.float64)
    r = np.linalg.norm(S, axis=1)
    Y = real_sh(J, S)                                  # [|S|, 2J+1]
    return radial(r, m, eps)[:, None, None] * np.einsum("sj,jab->sab", Y, Q)


VANISH_NORM = 1e-12


def normalise(B: np.ndarray) -> Optional[np.ndarray]:
    """Unit Frobenius norm, sign fixed by the first significant entry (row-major).

    An element that vanishes on the grid (norm below 1e-12; only J > 0 on a
    1x1x1 kernel, where Y^J(0) = 0) is dropped and yields None."""
    nrm = np.sqrt((B ** 2).sum())
    if nrm < VANISH_NORM:
        return None
    B = B / nrm
    flat = B.reshape(-1)
    first = flat[np.argmax(np.abs(flat) > SIGN_REL_THRESHOLD * np.abs(flat).max())]
    return B if first > 0 else -B


def j_range(k: int, l: int, jmax: Optional[int]) -> List[int]:
    top = k + l if jmax is None else min(k + l, jmax)
    return list(range(abs(k - l), top + 1))


def pair_basis(k: int, l: int, shells: Sequence[float], eps: float, ksize: int,
               jmax: Optional[int]) -> np.ndarray:
    """All normalised basis elements of the (k, l) block, ordered (J asc, shell): [nq, |S|, 2k+1, 2l+1].

    Elements that vanish on the grid are left out."""
    els = []
    for J in j_range(k, l, jmax):
        for m in shells:
            raw = raw_basis_kernel(k, l, J, m, eps, ksize)
            B = normalise(raw) if raw is not None else None
            if B is not None:
                els.append(B)
    return np.stack(els) if els else np.zeros((0, ksize ** 3, 2 * k + 1, 2 * l + 1))


def expand_fields(fields) -> List[Tuple[int, int]]:
    """Field list ((l, mult), ...) -> [(l, first channel)] per individual field, in channel order."""
    out, c = [], 0
    for l, mult in fields:
        for _ in range(mult):
            out.append((l, c))
            c += 2 * l + 1
    return out


def layer_basis(layer) -> Dict[Tuple[int, int], np.ndarray]:
    """Basis blocks for every (out order k, in order l) pair the layer uses."""
    ks = sorted({l for l, _ in layer.fields_out})
    ls = sorted({l for l, _ in layer.fields_in})
    return {(k, l): pair_basis(k, l, layer.shells, layer.eps, layer.ksize, layer.jmax)
            for k in ks for l in ls}


def coeff_count(layer) -> int:
    """Number of learned scalars: sum over (out field, in field) of the block's basis size.

    Without vanishing elements the block size is #shells * #J (Sec. 3.2.1)."""
    nq = {kl: B.shape[0] for kl, B in layer_basis(layer).items()}
    return sum(nq[(k, l)] for k, _ in expand_fields(layer.fields_out)
               for l, _ in expand_fields(layer.fields_in))


def paper_param_count(k: int, l: int, n_shells: int) -> int:
    """The paper's count of learnable parameters per (k, l) block: M (2 min(k, l) + 1)."""
    return n_shells * (2 * min(k, l) + 1)

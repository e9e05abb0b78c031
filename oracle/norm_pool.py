"""Steerable normalisation and sparse average pooling (oracle; test infrastructure only).

Norm (Sec. 3.3, Eq. 11): every irreducible field is normalised on its own,
with population statistics taken over all active sites of the tensor:
  l = 0 (one channel):   y = (f - E[f]) / sqrt(Var[f] + eps)
  l > 0 (2l+1 channels): y = f / sqrt(E[|f|^2] + eps)
so that multiplying a field by a scalar keeps its equivariance.

Pooling (the footnote of Sec. 3.1: downsampling is a stride-1 convolution
followed by average pooling, as in the cited 3D steerable CNNs): windows of
2x2x2 voxels with stride 2.  Output site x is active when some active input y
has floor(y / 2) = x; its value is the window's sum divided by 8, i.e. the
dense average pooling of the zero-filled grid, evaluated at active outputs.
Outputs are listed in lexicographic (b, x, y, z) order.

Readings where the paper is silent:
  * eps = 1e-5;
  * the population is every active site of every batch entry (training-mode
    statistics), and Var is the population (biased) variance;
  * no affine parameters after the normalisation (the paper shows none);
  * pooling divides by the window volume 8 (dense semantics of the cited
    method), not by the number of active inputs.

Everything is fp64 numpy.
"""
from typing import List, Tuple

import numpy as np

EPS = 1e-5


def _field_slices(fields) -> List[Tuple[int, int, int]]:
    """[(l, first channel, channel count)] for a field list ((l, multiplicity), ...)."""
    out, c = [], 0
    for l, m in fields:
        for _ in range(m):
            out.append((l, c, 2 * l + 1))
            c += 2 * l + 1
    return out


def norm_forward(x: np.ndarray, fields, eps: float = EPS) -> np.ndarray:
    """Eq. 11 applied field by field over the rows of x ([N, C])."""
    x = np.asarray(x, np.float64)
    y = np.empty_like(x)
    for l, c, d in _field_slices(fields):
        f = x[:, c:c + d]
        if l == 0:
            y[:, c:c + d] = (f - f.mean()) / np.sqrt(f.var() + eps)
        else:
            y[:, c:c + d] = f / np.sqrt((f * f).sum(1).mean() + eps)
    return y


def norm_backward(x: np.ndarray, dy: np.ndarray, fields, eps: float = EPS) -> np.ndarray:
    """Gradient of <norm_forward(x), dy> with respect to x (the statistics depend on x)."""
    x = np.asarray(x, np.float64)
    dy = np.asarray(dy, np.float64)
    n = x.shape[0]
    dx = np.empty_like(x)
    for l, c, d in _field_slices(fields):
        f, g = x[:, c:c + d], dy[:, c:c + d]
        if l == 0:
            r = 1.0 / np.sqrt(f.var() + eps)
            xh = (f - f.mean()) * r
            dx[:, c:c + d] = r * (g - g.mean() - xh * (g * xh).mean())
        else:
            nu = (f * f).sum(1).mean()
            r = 1.0 / np.sqrt(nu + eps)
            dx[:, c:c + d] = r * g - (r ** 3 / n) * (g * f).sum() * f
    return dx


def pool_sites(coords: np.ndarray) -> np.ndarray:
    """Output sites of 2x2x2 / stride-2 pooling: the distinct (b, floor(x/2), floor(y/2), floor(z/2)),
    lexicographic."""
    c = np.asarray(coords, np.int64).reshape(-1, 4)
    o = c.copy()
    o[:, 1:] //= 2
    return np.unique(o, axis=0).astype(np.int32) if len(o) else np.zeros((0, 4), np.int32)


def pool_members(coords_in: np.ndarray, coords_out: np.ndarray) -> np.ndarray:
    """[N_in] output row of each input site (the window it falls in)."""
    cin = np.asarray(coords_in, np.int64).reshape(-1, 4)
    H = {tuple(int(v) for v in c): r for r, c in enumerate(np.asarray(coords_out, np.int64))}
    out = np.empty(len(cin), np.int64)
    for r, c in enumerate(cin):
        out[r] = H[(int(c[0]), int(c[1]) // 2, int(c[2]) // 2, int(c[3]) // 2)]
    return out


def pool_forward(x: np.ndarray, member: np.ndarray, n_out: int) -> np.ndarray:
    """Window sums / 8."""
    y = np.zeros((n_out, x.shape[1]))
    np.add.at(y, member, np.asarray(x, np.float64))
    return y / 8.0


def pool_backward(dy: np.ndarray, member: np.ndarray) -> np.ndarray:
    """Adjoint of pool_forward: every input receives its window's gradient / 8."""
    return np.asarray(dy, np.float64)[member] / 8.0


def dense_avg_pool(coords: np.ndarray, x: np.ndarray, grid: int, batch: int) -> np.ndarray:
    """Zero-filled dense grid [B, G, G, G, C] averaged over 2x2x2 blocks (G even)."""
    assert grid % 2 == 0
    C = x.shape[1]
    g = np.zeros((batch, grid, grid, grid, C))
    c = np.asarray(coords, np.int64)
    g[c[:, 0], c[:, 1], c[:, 2], c[:, 3]] = x
    h = grid // 2
    return g.reshape(batch, h, 2, h, 2, h, 2, C).mean(axis=(2, 4, 6))

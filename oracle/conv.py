"""Kernel synthesis, sparse steerable convolution and its adjoint (oracle; test infrastructure only).

* ``synth``      Eq. 7 per (out field, in field) block, assembled as the block
                 matrix of Eq. 9: kappa(s) in R^{K_out x K_in} for every offset.
* ``forward``    Alg. 1, feature update: F_out starts at zero and, for every
                 offset s and pair (o, i) in R_s, F_out[o] += kappa(s) F_in[i].
* ``backward``   the exact adjoint of ``forward`` and ``synth`` (the paper does
                 not state a backward pass): dF_in, dkappa and the gradient of
                 the learned coefficients w.
* ``dense_conv`` Eq. 1 / Eq. 6 evaluated on the densified voxel grid by shifted
                 array sums (independent of any rule book), used to pin
                 ``forward``.
* ``gate_forward`` / ``gate_backward``  the nonlinearity of Sec. 3.3 (Eq. 12):
                 ReLU on l = 0 fields and Sigmoid(gate) * f on l > 0 fields, the
                 gate being an extra scalar output channel of the same SS-Conv
                 (one per l > 0 field, appended after the fields in field order).
                 ReLU'(0) is taken as 0.

Channel layout (Sec. 3.1, Eq. 5): fields in list order, each field's 2l+1
components contiguous (j = -l..l).  All arithmetic is fp64.
"""
from typing import Dict, List, Tuple

import numpy as np

from .basis import expand_fields, layer_basis, offsets


def coeff_blocks(layer, basis: Dict[Tuple[int, int], np.ndarray]):
    """Yield (out row offset, k, in col offset, l, coefficient offset, nq) in coefficient order.

    Coefficients are ordered by (out field, in field, J, shell)."""
    off = 0
    for k, ro in expand_fields(layer.fields_out):
        for l, ci in expand_fields(layer.fields_in):
            nq = basis[(k, l)].shape[0]
            yield ro, k, ci, l, off, nq
            off += nq


def synth(layer, basis, coeffs: np.ndarray) -> np.ndarray:
    """kappa [|S|, Cout, Cin] = sum_q w_q B_q per block (Eq. 7, Eq. 9)."""
    w = np.asarray(coeffs, np.float64)
    kap = np.zeros((layer.ksize ** 3, layer.cout, layer.cin))
    for ro, k, ci, l, off, nq in coeff_blocks(layer, basis):
        kap[:, ro:ro + 2 * k + 1, ci:ci + 2 * l + 1] = np.einsum("q,qsab->sab", w[off:off + nq], basis[(k, l)])
    return kap


def synth_adjoint(layer, basis, dkappa: np.ndarray) -> np.ndarray:
    """d w_q = sum_s <dkappa[s] block, B_q[s]>_F, the adjoint of ``synth``."""
    n = sum(nq for *_, nq in coeff_blocks(layer, basis))
    dw = np.zeros(n)
    for ro, k, ci, l, off, nq in coeff_blocks(layer, basis):
        blk = dkappa[:, ro:ro + 2 * k + 1, ci:ci + 2 * l + 1]
        dw[off:off + nq] = np.einsum("sab,qsab->q", blk, basis[(k, l)])
    return dw


def _unique(idx: np.ndarray) -> np.ndarray:
    # Within one R_s an output row pairs with at most one input row (y = stride*x - s)
    # and vice versa, so a buffered fancy-index update adds every pair exactly once.
    assert len(np.unique(idx)) == len(idx), "rule book offset lists must not repeat a row"
    return idx


def forward(feats_in: np.ndarray, R: List[np.ndarray], kappa: np.ndarray, n_out: int) -> np.ndarray:
    """F_out[o] += kappa(s) F_in[i] for every (o, i) in every R_s; F_out starts at zero."""
    f = np.asarray(feats_in, np.float64)
    out = np.zeros((n_out, kappa.shape[1]))
    for si, r in enumerate(R):
        if len(r):
            out[_unique(r[:, 0])] += f[r[:, 1]] @ kappa[si].T
    return out


def forward_loop(feats_in, R, kappa, n_out):
    """The same update written as the explicit pair loop (tiny inputs)."""
    f = np.asarray(feats_in, np.float64)
    out = np.zeros((n_out, kappa.shape[1]))
    for si, r in enumerate(R):
        for o, i in r:
            out[o] += kappa[si] @ f[i]
    return out


def forward_rows(feats_in, nbr: np.ndarray, kappa, rows: np.ndarray) -> np.ndarray:
    """F_out at selected output rows only, from the neighbour map nbr[s, out row]."""
    f = np.asarray(feats_in, np.float64)
    out = np.zeros((len(rows), kappa.shape[1]))
    for si in range(kappa.shape[0]):
        src = nbr[si, rows]
        hit = src >= 0
        if hit.any():
            out[hit] += f[src[hit]] @ kappa[si].T
    return out


def grad_feats(grad_out, R, kappa, n_in):
    """dF_in[i] = sum_s sum_{(o, i) in R_s} kappa(s)^T grad_out[o] (adjoint of ``forward``)."""
    g = np.asarray(grad_out, np.float64)
    d_in = np.zeros((n_in, kappa.shape[2]))
    for si, r in enumerate(R):
        if len(r):
            d_in[_unique(r[:, 1])] += g[r[:, 0]] @ kappa[si]
    return d_in


def grad_kappa(feats_in, grad_out, R, kappa_shape):
    """dkappa(s) = sum_{(o, i) in R_s} grad_out[o] F_in[i]^T."""
    f = np.asarray(feats_in, np.float64)
    g = np.asarray(grad_out, np.float64)
    dk = np.zeros(kappa_shape)
    for si, r in enumerate(R):
        if len(r):
            dk[si] = g[r[:, 0]].T @ f[r[:, 1]]
    return dk


def backward(feats_in, grad_out, R, kappa, n_in):
    """(dF_in [n_in, Cin], dkappa [|S|, Cout, Cin]) for L = <F_out, grad_out>."""
    return grad_feats(grad_out, R, kappa, n_in), grad_kappa(feats_in, grad_out, R, kappa.shape)


def dense_conv(coords_in, feats_in, kappa, grid: int, stride: int, batch: int) -> np.ndarray:
    """Eq. 6 without the site-state rule: out[b, x] = sum_s kappa(s) f_dense[b, stride*x - s].

    Returns the dense output [batch, G, G, G, Cout] with G = ceil(grid/stride).
    """
    ksize = round(kappa.shape[0] ** (1 / 3))
    h = (ksize - 1) // 2
    c = np.asarray(coords_in, np.int64)
    cin = kappa.shape[2]
    dense = np.zeros((batch, grid + 2 * h, grid + 2 * h, grid + 2 * h, cin))
    dense[c[:, 0], c[:, 1] + h, c[:, 2] + h, c[:, 3] + h] = feats_in
    G = -(-grid // stride)
    out = np.zeros((batch, G, G, G, kappa.shape[1]))
    for si, s in enumerate(offsets(ksize)):
        lo = h - s                                    # padded index of stride*0 - s
        sl = tuple(slice(lo[a], lo[a] + stride * (G - 1) + 1, stride) for a in range(3))
        window = dense[(slice(None),) + sl]           # [B, G', G', G', Cin], may be short at the far edge
        gx, gy, gz = window.shape[1:4]
        out[:, :gx, :gy, :gz] += window @ kappa[si].T
    return out


# ----------------------------------------------------------------------------
# gated nonlinearity (Sec. 3.3, Eq. 12)
# ----------------------------------------------------------------------------

def _gate_plan(fields):
    """[(l, channel offset, gate channel or -1)] for each regular field; gates follow the fields."""
    plan = []
    c = 0
    for l, m in fields:
        for _ in range(m):
            plan.append([l, c, -1])
            c += 2 * l + 1
    g = c
    for p in plan:
        if p[0] > 0:
            p[2] = g
            g += 1
    return plan, c, g


def sigmoid(x):
    return 1.0 / (1.0 + np.exp(-x))


def gate_forward(x: np.ndarray, fields) -> np.ndarray:
    """[N, C + n_gates] -> [N, C]: ReLU on scalars, Sigmoid(gate) * f on l > 0 fields."""
    plan, c, g = _gate_plan(fields)
    assert x.shape[1] == g
    y = np.zeros((x.shape[0], c))
    for l, o, gc in plan:
        if l == 0:
            y[:, o] = np.maximum(x[:, o], 0.0)
        else:
            y[:, o:o + 2 * l + 1] = sigmoid(x[:, gc:gc + 1]) * x[:, o:o + 2 * l + 1]
    return y


def gate_backward(x: np.ndarray, dy: np.ndarray, fields) -> np.ndarray:
    plan, c, g = _gate_plan(fields)
    dx = np.zeros_like(x, dtype=np.float64)
    for l, o, gc in plan:
        if l == 0:
            dx[:, o] = dy[:, o] * (x[:, o] > 0)
        else:
            sg = sigmoid(x[:, gc])
            f = x[:, o:o + 2 * l + 1]
            d = dy[:, o:o + 2 * l + 1]
            dx[:, o:o + 2 * l + 1] = d * sg[:, None]
            dx[:, gc] = (d * f).sum(1) * sg * (1 - sg)
    return dx


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round to the nearest bfloat16 value (ties to even), as float64 (the bf16 kernel's precision)."""
    f = np.ascontiguousarray(x, np.float32)
    b = f.view(np.uint32).astype(np.uint64)
    r = (((b + 0x7FFF + ((b >> 16) & 1)) >> 16) << 16).astype(np.uint32)
    return r.view(np.float32).astype(np.float64).reshape(np.shape(x))


class Layer:
    """Everything the oracle needs for one SS-Conv layer (basis built once)."""

    def __init__(self, spec):
        self.spec = spec
        self.basis = layer_basis(spec)
        self.n_coeff = sum(nq for *_, nq in coeff_blocks(spec, self.basis))

    def kappa(self, coeffs, bf16=False):
        k = synth(self.spec, self.basis, coeffs)
        return round_bf16(k) if bf16 else k

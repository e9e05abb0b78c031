"""Seeded parity cases: inputs from ``workloads`` and fp64 expectations from ``oracle``.

Shared by the GPU parity tests and the smoke check; nothing here calls the HIP
library.
"""
from dataclasses import dataclass
from functools import lru_cache
from typing import List

import numpy as np

from oracle import conv as oc
from oracle import rulebook as orb
from workloads import CONFIGS
from workloads.gen import make_coeffs, make_coords, make_features, make_grad


def rel_err(got, want) -> float:
    """L_inf error over the L_inf norm of the expectation."""
    want = np.asarray(want, np.float64)
    return float(np.abs(np.asarray(got, np.float64) - want).max() / max(np.abs(want).max(), 1e-300))


@dataclass
class LayerRef:
    spec: object
    grid: int
    coords_in: np.ndarray
    coords_out: np.ndarray
    R: List[np.ndarray]
    nbr: np.ndarray
    lay: oc.Layer
    coeffs: np.ndarray
    kappa: np.ndarray        # fp64 (bf16-rounded for bf16 workloads)


@lru_cache(maxsize=None)
def coords_of(i: int) -> np.ndarray:
    return make_coords(CONFIGS[i])


@lru_cache(maxsize=None)
def layers_of(i: int):
    """Oracle rule books and kernels of every layer of workload i (no features)."""
    spec = CONFIGS[i]
    lays = [oc.Layer(L) for L in spec.layers]
    coeffs = make_coeffs(spec, [l.n_coeff for l in lays])
    bf16 = spec.dtype == "bf16"
    out, c, g = [], coords_of(i), spec.grid
    for L, lay, w in zip(spec.layers, lays, coeffs):
        co = orb.output_sites(c, g, L.ksize, L.stride, L.submanifold)
        R = orb.rulebook(c, co, L.ksize, L.stride)
        out.append(LayerRef(L, g, c, co, R, orb.neighbour_map(R, len(co)), lay, w, lay.kappa(w, bf16=bf16)))
        c, g = co, -(-g // L.stride)
    return out


@lru_cache(maxsize=None)
def features_of(i: int) -> np.ndarray:
    spec = CONFIGS[i]
    return make_features(spec, len(coords_of(i)), spec.layers[0].cin)


@lru_cache(maxsize=None)
def single_layer_reference(i: int):
    """(out, grad_out, grad_feats, grad_coeffs) of the first layer of workload i, fp64."""
    spec = CONFIGS[i]
    L = layers_of(i)[0]
    f = features_of(i)
    out = oc.forward(f, L.R, L.kappa, len(L.coords_out))
    g = make_grad(spec, len(L.coords_out), L.spec.cout)
    d_in = oc.grad_feats(g, L.R, L.kappa, len(f))
    dk = oc.grad_kappa(f, g, L.R, L.kappa.shape)
    dw = oc.synth_adjoint(L.spec, L.lay.basis, dk)
    return out, g, d_in, dw


@lru_cache(maxsize=None)
def stack_reference(i: int):
    """Forward features of every layer and the gradients of the whole stack (fp64)."""
    spec = CONFIGS[i]
    Ls = layers_of(i)
    h = features_of(i).astype(np.float64)
    xs, ys = [], []
    for L in Ls:
        xs.append(h)
        y = oc.forward(h, L.R, L.kappa, len(L.coords_out))
        ys.append(y)
        h = oc.gate_forward(y, L.spec.fields_out[:-1]) if L.spec.gated else y
    g = make_grad(spec, len(Ls[-1].coords_out), Ls[-1].spec.cout).astype(np.float64)
    grads = [None] * len(Ls)
    for idx in range(len(Ls) - 1, -1, -1):
        L = Ls[idx]
        if L.spec.gated:
            g = oc.gate_backward(ys[idx], g, L.spec.fields_out[:-1])
        dk = oc.grad_kappa(xs[idx], g, L.R, L.kappa.shape)
        grads[idx] = oc.synth_adjoint(L.spec, L.lay.basis, dk)
        g = oc.grad_feats(g, L.R, L.kappa, len(L.coords_in))
    return xs, ys, h, g, grads


@lru_cache(maxsize=None)
def block_reference(i: int):
    """The downsampling block of workload i in fp64: SS-Conv -> Norm -> gate -> average pooling.

    Returns (pooled coords, pooled output, upstream gradient, grad of the block input,
    grad of the coefficients)."""
    from oracle import norm_pool as onp
    spec = CONFIGS[i]
    L = layers_of(i)[0]
    f = features_of(i).astype(np.float64)
    fo = L.spec.fields_out
    regular = fo[:-1] if L.spec.gated else fo
    y = oc.forward(f, L.R, L.kappa, len(L.coords_out))
    z = onp.norm_forward(y, fo)
    h = oc.gate_forward(z, regular) if L.spec.gated else z
    pc = onp.pool_sites(L.coords_out)
    member = onp.pool_members(L.coords_out, pc)
    out = onp.pool_forward(h, member, len(pc))
    g = make_grad(spec, len(pc), h.shape[1]).astype(np.float64)
    gh = onp.pool_backward(g, member)
    gz = oc.gate_backward(z, gh, regular) if L.spec.gated else gh
    gy = onp.norm_backward(y, gz, fo)
    d_in = oc.grad_feats(gy, L.R, L.kappa, len(f))
    dk = oc.grad_kappa(f, gy, L.R, L.kappa.shape)
    dw = oc.synth_adjoint(L.spec, L.lay.basis, dk)
    return pc, out, g, d_in, dw

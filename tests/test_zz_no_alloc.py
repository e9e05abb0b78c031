"""The allocation-free forward (ssconv_forward_noalloc) against ssconv_forward.

Both entry points are called through the C ABI on the same seeded inputs, twice
in a row per layer shape, the second time on a smaller input (a prefix of the
sites), so the second call runs on scratch the first one left behind.  Where
the two calls take the same kernels (every bf16 layer; fp32 layers whose
scratch fits the fixed region) the outputs must be bit-identical; a sparse fp32
layer whose pair-list buffers exceed the region runs the output-stationary
kernel instead and must agree within the fp32 parity tolerance (1e-4 of the
L_inf norm).  A bf16 kernel too large for the region must be rejected with an
error, leaving the output untouched.
"""
import numpy as np
import pytest

from workloads import CONFIGS
from workloads.configs import LayerSpec
from workloads.gen import make_coeffs, make_coords, make_features

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
P = pytest.importorskip("paper_2111_07383_amd")

DEV = "cuda:0"


def _rel(a, b):
    a = a.double().cpu().numpy()
    b = b.double().cpu().numpy()
    return float(np.abs(a - b).max() / max(np.abs(b).max(), 1e-300))


def _layer(L, dtype, seed_cfg):
    desc = P.layer_desc(L)
    basis = torch.from_numpy(P.basis_build(desc)).to(DEV)
    n_coeff = P.basis_info(desc)[1]
    coeffs = torch.from_numpy(make_coeffs(seed_cfg, [n_coeff])[0]).to(DEV)
    return P.synth_kernel(desc, basis, coeffs, dtype)


def _both(coords, grid, L, W, feats):
    rb = P.Rulebook(coords, grid, L.ksize, L.stride, L.submanifold)
    want = P.forward(feats, rb, W)
    got = torch.full_like(want, float("nan"))
    P.forward_noalloc(feats, rb, W, got)
    torch.cuda.synchronize()
    rb.close()
    return got, want


# (workload, layer index, rows of the second, smaller call, exact): the bf16 208-channel 128^3
# layer; the fp32 104-channel 5^3 layer; the sparse stride-2 fp32 layer (pair-list path, its
# buffers fit the region); layer 2 of the stack (5^3, 104 -> 256 fp32: its pair-list buffers do
# not fit, so the output-stationary kernel runs and only the tolerance applies)
CASES = [(4, 0, 20000, True), (2, 0, 6000, True), (3, 0, 9000, True), (5, 1, 8000, False)]


@pytest.mark.parametrize("i,layer,small,exact", CASES)
def test_noalloc_forward_matches_forward_twice(i, layer, small, exact):
    spec = CONFIGS[i]
    L = spec.layers[layer]
    dt = torch.bfloat16 if spec.dtype == "bf16" else torch.float32
    coords = torch.from_numpy(make_coords(spec)).to(DEV)
    W = _layer(L, dt, spec)
    for n in (int(coords.shape[0]), small):
        print(f"noalloc forward: workload {i} layer {layer} rows {n} dtype {spec.dtype}", flush=True)
        feats = torch.from_numpy(make_features(spec, n, L.cin)).to(DEV).to(dt)
        got, want = _both(coords[:n].contiguous(), spec.grid, L, W, feats)
        assert not torch.isnan(got.float()).any()
        if exact:
            assert torch.equal(got, want), _rel(got, want)
        else:
            assert _rel(got, want) <= 1e-4


def test_noalloc_rejects_a_kernel_beyond_its_scratch():
    # bf16, 3x3x3, 1120 -> 1120 scalar channels: the packed kernel needs 2 * 27 * 1120^2 bytes,
    # more than the fixed region holds
    assert 2 * 27 * 1120 * 1120 > P.NOALLOC_SCRATCH_BYTES
    L = LayerSpec(3, 1, True, ((0, 1120),), ((0, 1120),), shells=(0.0, 1.0))
    coords = torch.tensor([[0, 1, 1, 1], [0, 1, 1, 2], [0, 2, 1, 1]], dtype=torch.int32, device=DEV)
    rb = P.Rulebook(coords, 8, 3, 1, True)
    W = torch.zeros((27, 1120, 1120), dtype=torch.bfloat16, device=DEV)
    feats = torch.ones((3, 1120), dtype=torch.bfloat16, device=DEV)
    out = torch.full((3, 1120), 7.0, dtype=torch.bfloat16, device=DEV)
    with pytest.raises(P.SSConvError, match="scratch"):
        P.forward_noalloc(feats, rb, W, out)
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())
    rb.close()
    del L

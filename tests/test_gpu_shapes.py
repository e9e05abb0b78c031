"""GPU parity of the convolution kernels (gather GEMM, Sec. 3.2.3 Alg. 1 feature update; its
adjoints: the feature gradient on the mirrored or inverted map, the kernel gradient and the
synthesis adjoint) on shapes beyond the workloads' layers: every column-block width of the bf16
gather kernel (4, 8, 13 and 14 blocks of 16), output channels that leave a partial block, two
column tiles, a stride-2 layer on a generated output set, a 1^3 kernel, several batch entries,
and a dense 196 608-site set.  bf16, and fp32 both as the cost model chooses (pair lists or the
output-stationary kernel) and with the pair-list path forbidden (override 10).  Against the
fp64 oracle on the exact inputs (bf16-rounded for bf16) within 2e-2 (bf16) or 1e-4 (fp32) of
the L_inf norm; every call goes through the C ABI.
"""
import numpy as np
import pytest

from cases import layers_of, rel_err
from oracle import conv as oc
from oracle import rulebook as orb
from workloads.configs import LayerSpec

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
P = pytest.importorskip("paper_2111_07383_amd")

DEV = "cuda:0"
TOL = {"bf16": 2e-2, "f32": 1e-4}


def _dev(a, dt):
    """(tensor of dtype dt on the device, its fp64 values)."""
    t = torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(dt)
    return t.to(DEV), t.double().numpy()


def _coords(seed, n, grid, batch=1):
    rng = np.random.default_rng(seed)
    c = np.concatenate([rng.integers(0, batch, (n, 1)), rng.integers(0, grid, (n, 3))], 1)
    return np.unique(c, axis=0).astype(np.int32)


def _layer(coords, grid, spec, seed, label, dtype="bf16", variant=0):
    """Synthesised layer (fields of spec): forward, feature and coefficient gradients."""
    label = f"{label}, {dtype}" + (f", override {variant}" if variant else "")
    print(label, flush=True)
    dt = torch.bfloat16 if dtype == "bf16" else torch.float32
    rng = np.random.default_rng(seed)
    lay = oc.Layer(spec)
    w = rng.standard_normal(lay.n_coeff).astype(np.float32)
    x_t, x = _dev(rng.standard_normal((len(coords), spec.cin)), dt)
    co = orb.output_sites(coords, grid, spec.ksize, spec.stride, spec.submanifold)
    R = orb.rulebook(coords, co, spec.ksize, spec.stride)
    g_t, g = _dev(rng.standard_normal((len(co), spec.cout)), dt)
    kap = lay.kappa(w, bf16=(dtype == "bf16"))
    want = oc.forward(x, R, kap, len(co))
    want_gf = oc.grad_feats(g, R, kap, len(coords))
    want_gc = oc.synth_adjoint(spec, lay.basis, oc.grad_kappa(x, g, R, kap.shape))
    desc = P.layer_desc(spec)
    basis = torch.from_numpy(P.basis_build(desc)).to(DEV)
    rb = P.Rulebook(torch.from_numpy(coords).to(DEV), grid, spec.ksize, spec.stride, spec.submanifold)
    W = P.synth_kernel(desc, basis, torch.from_numpy(w).to(DEV), dt)
    P.debug_set(3, variant)
    try:
        y = P.forward(x_t, rb, W)
        gf, gc = P.backward(x_t, g_t, rb, W, desc, basis)
        torch.cuda.synchronize()
    finally:
        P.debug_set(3, 0)
    rb.close()
    errs = (rel_err(y.double().cpu().numpy(), want), rel_err(gf.double().cpu().numpy(), want_gf),
            rel_err(gc.double().cpu().numpy(), want_gc))
    print(f"{label}: forward {errs[0]:.2e}, grad_feats {errs[1]:.2e}, grad_coeffs {errs[2]:.2e}", flush=True)
    assert max(errs) < TOL[dtype]


# (ksize, stride, submanifold, fields in, fields out): channel counts in the comment
SHAPES = {
    "w8_32to80": (3, 1, True, ((0, 8), (1, 8)), ((0, 16), (1, 8), (2, 8))),          # 32 -> 80: 5 of 8 blocks
    "w4_16to24": (3, 1, True, ((0, 16),), ((0, 9), (1, 5))),                         # 16 -> 24: 2 of 4 blocks
    "w13_24to300": (3, 1, True, ((0, 24),), ((0, 100), (1, 40), (2, 16))),          # 24 -> 300: two tiles of 10 blocks
    "w14_32to224": (3, 1, True, ((0, 8), (1, 8)), ((0, 224),)),                     # 32 -> 224: 14 blocks
    "ragged_40to9": (3, 1, True, ((0, 40),), ((0, 6), (1, 1))),                     # 40 -> 9: a partial block
    "k1_64to80": (1, 1, True, ((0, 16), (1, 16)), ((0, 32), (1, 16))),              # 1^3 kernel
    "s2_32to72": (3, 2, False, ((0, 8), (1, 8)), ((0, 8), (1, 8), (2, 8))),         # stride 2, inverted map
}


MODES = [("bf16", 0), ("f32", 0), ("f32", 10)]


def _spec(name):
    k, st, sub, fin, fout = SHAPES[name]
    return LayerSpec(k, st, sub, fin, fout, shells=tuple(float(m) for m in range(k // 2 + 1)))


@pytest.mark.parametrize("dtype,variant", MODES)
@pytest.mark.parametrize("name", list(SHAPES))
def test_layer_shapes_objects(name, dtype, variant):
    """The sparse objects of the downsampling workload (32 batch entries, 64^3)."""
    L = layers_of(6)[0]
    _layer(L.coords_in, L.grid, _spec(name), len(name), f"objects, {name}", dtype, variant)


@pytest.mark.parametrize("dtype,variant", MODES)
@pytest.mark.parametrize("name", ["w8_32to80", "s2_32to72", "ragged_40to9"])
def test_layer_shapes_small(name, dtype, variant):
    """333 random sites in a 12^3 grid over 3 batch entries: two row tiles, the second partial."""
    _layer(_coords(11, 400, 12, batch=3), 12, _spec(name), 3, f"small, {name}", dtype, variant)


@pytest.mark.parametrize("dtype,variant", MODES)
def test_dense_slabs(dtype, variant):
    """Three dense 256 x 256 slabs (196 608 sites, 3^3 submanifold, 8 -> 8 scalar channels): every
    tile's neighbour rows lie ~65 536 rows apart."""
    x, y, z = np.meshgrid(np.arange(3), np.arange(256), np.arange(256), indexing="ij")
    c = np.stack([np.zeros(x.size, np.int64), x.ravel(), y.ravel(), z.ravel()], 1).astype(np.int32)
    spec = LayerSpec(3, 1, True, ((0, 8),), ((0, 8),), shells=(0.0, 1.0))
    _layer(c, 256, spec, 1, "dense slabs", dtype, variant)

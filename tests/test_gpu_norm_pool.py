"""GPU parity of the steerable normalisation (Sec. 3.3, Eq. 11), the 2x2x2 average pooling
(footnote of Sec. 3.1) and the downsampling block built from them, against the fp64 oracle.

Pooling rule books must match the oracle exactly (output sites, window membership, offset of
every member); features within 1e-4 (fp32) or 2e-2 (bf16) as L_inf error over the L_inf norm of
the oracle result.  Every call goes through the C ABI.
"""
import numpy as np
import pytest

from cases import block_reference, coords_of, features_of, layers_of, rel_err
from oracle import norm_pool as onp
from workloads import CONFIGS
from workloads.gen import round_bf16

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
P = pytest.importorskip("paper_2111_07383_amd")
from paper_2111_07383_amd import _abi  # noqa: E402
from paper_2111_07383_amd.stack import DownBlock  # noqa: E402

DEV = "cuda:0"
TOL = {torch.float32: 1e-4, torch.bfloat16: 2e-2}


def _tensor(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
    return t.to(dtype) if dtype is not None else t


def _inputs(rng, n, C, dtype, shift=0.0):
    x = (rng.standard_normal((n, C)) * rng.uniform(0.5, 2.0, C) + shift).astype(np.float32)
    if dtype == torch.bfloat16:
        x = round_bf16(x)
    return x


def _random_sites(rng, n, grid, batch):
    c = np.stack([rng.integers(0, batch, n), rng.integers(0, grid, n), rng.integers(0, grid, n),
                  rng.integers(0, grid, n)], 1)
    return np.unique(c, axis=0).astype(np.int32)


# ---- pooling rule book -------------------------------------------------------------------

def _pool_cases():
    rng = np.random.default_rng(20211107)
    return {
        "objects64_b32": (coords_of(6), 64),
        "sphere16": (coords_of(1), 16),
        "odd_grid5": (_random_sites(rng, 60, 5, 2), 5),        # ceil(5/2) = 3 per axis
        "dense_cube8": (np.stack(np.meshgrid([0], *[np.arange(8)] * 3, indexing="ij"), -1)
                        .reshape(-1, 4).astype(np.int32), 8),   # every window full
        "single": (np.array([[0, 3, 4, 5]], np.int32), 7),
    }


@pytest.mark.parametrize("name", ["objects64_b32", "sphere16", "odd_grid5", "dense_cube8", "single"])
def test_pool_rulebook_exact(name):
    coords, grid = _pool_cases()[name]
    print(f"pool rule book {name} n={len(coords)} grid {grid}", flush=True)
    rb = P.Rulebook(_tensor(coords), grid, 2, 2, False)
    want = onp.pool_sites(coords)
    np.testing.assert_array_equal(rb.out_coords().cpu().numpy(), want)
    member = onp.pool_members(coords, want)
    nbr = rb.neighbours().cpu().numpy()                     # [8, n_out]
    assert nbr.shape == (8, len(want))
    s_idx, o = np.nonzero(nbr >= 0)
    i = nbr[s_idx, o]
    # every input appears exactly once, in its own window, at the offset 2x - y
    assert len(i) == len(coords) and len(np.unique(i)) == len(coords)
    np.testing.assert_array_equal(member[i], o)
    d = 2 * want[o, 1:].astype(np.int64) - coords[i, 1:]     # in {-1, 0}^3
    np.testing.assert_array_equal(((d[:, 0] + 1) * 2 + (d[:, 1] + 1)) * 2 + (d[:, 2] + 1), s_idx)
    assert rb.n_pairs == len(coords)
    rb.close()


def test_pool_rulebook_empty():
    rb = P.Rulebook(torch.zeros((0, 4), dtype=torch.int32, device=DEV), 8, 2, 2, False)
    assert rb.n_out == 0 and rb.n_pairs == 0
    out = P.pool_forward(torch.zeros((0, 5), device=DEV), rb)
    assert out.shape == (0, 5)
    rb.close()


# ---- pooling forward / backward -----------------------------------------------------------

@pytest.mark.parametrize("name,C,dtype", [("objects64_b32", 144, torch.float32), ("objects64_b32", 120, torch.bfloat16),
                                          ("odd_grid5", 7, torch.float32), ("odd_grid5", 5, torch.bfloat16),
                                          ("dense_cube8", 16, torch.float32), ("single", 3, torch.float32)])
def test_pool_forward_backward(name, C, dtype):
    coords, grid = _pool_cases()[name]
    print(f"pool {name} C={C} {dtype}", flush=True)
    rng = np.random.default_rng(7 + C)
    x = _inputs(rng, len(coords), C, dtype)
    rb = P.Rulebook(_tensor(coords), grid, 2, 2, False)
    pc = onp.pool_sites(coords)
    member = onp.pool_members(coords, pc)
    g = _inputs(rng, len(pc), C, dtype)
    y = P.pool_forward(_tensor(x, dtype), rb).float().cpu().numpy()
    dx = P.pool_backward(_tensor(g, dtype), rb).float().cpu().numpy()
    assert rel_err(y, onp.pool_forward(x, member, len(pc))) < TOL[dtype]
    assert rel_err(dx, onp.pool_backward(g, member)) < TOL[dtype]
    if dtype == torch.float32:
        # fp32 sums of at most 8 values, scaled by 1/8: within a few ulps
        assert rel_err(y, onp.pool_forward(x, member, len(pc))) < 1e-6
        np.testing.assert_array_equal(dx, (g / np.float32(8))[member])
    rb.close()


# ---- norm --------------------------------------------------------------------------------

NORM_CASES = {
    "objects_block": (((0, 32), (1, 16), (2, 8), (0, 24)), 3001),   # C = 144, 1 row group of 144
    "mixed_small": (((0, 2), (1, 1), (2, 1)), 7),                 # C = 10, 25 row groups, ragged
    "scalar_one": (((0, 1),), 5000),                               # C = 1, 256 row groups
    "wide": (((0, 64), (1, 64), (2, 32)), 1500),                   # C = 416 > 256: two channel chunks
    "vectors_only": (((1, 3), (3, 2)), 999),                       # C = 23, no scalar field
    "single_row": (((0, 3), (1, 2)), 1),                           # var = 0: scalars become 0
    "max_channels": (((0, 64), (1, 64), (2, 64), (3, 32), (4, 16), (0, 80)), 777),  # C = 1024
    "fp32_vectors": (((0, 4), (1, 1), (2, 1)), 4097),             # C = 12: 16-byte vectors in fp32 only
}


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("name", list(NORM_CASES))
def test_norm_forward_backward(name, dtype):
    fields, n = NORM_CASES[name]
    C = P.n_channels(fields)
    print(f"norm {name} n={n} C={C} {dtype}", flush=True)
    rng = np.random.default_rng(n + C)
    x = _inputs(rng, n, C, dtype, shift=0.3)
    g = _inputs(rng, n, C, dtype)
    y = P.norm_forward(fields, _tensor(x, dtype)).float().cpu().numpy()
    dx = P.norm_backward(fields, _tensor(x, dtype), _tensor(g, dtype)).float().cpu().numpy()
    wy, wdx = onp.norm_forward(x, fields), onp.norm_backward(x, g, fields)
    e1, e2 = rel_err(y, wy), rel_err(dx, wdx)
    print(f"norm {name} {dtype} errors {e1:.3e} {e2:.3e}", flush=True)
    assert e1 < TOL[dtype] and e2 < TOL[dtype]


def test_norm_large_mean_and_in_place():
    """Scalar fields far from zero (mean 1000, std ~1): fp64 sums keep the variance exact; the
    output may overwrite the input."""
    fields = ((0, 8), (1, 4))
    rng = np.random.default_rng(11)
    x = _inputs(rng, 4096, 20, torch.float32)
    x[:, :8] += 1000.0
    g = _inputs(rng, 4096, 20, torch.float32)
    xt = _tensor(x)
    dx = P.norm_backward(fields, xt, _tensor(g)).cpu().numpy()
    assert rel_err(dx, onp.norm_backward(x, g, fields)) < 1e-4
    P.norm_forward(fields, xt, out=xt)
    assert rel_err(xt.cpu().numpy(), onp.norm_forward(x, fields)) < 1e-4


def test_norm_deterministic():
    fields, n = NORM_CASES["objects_block"]
    rng = np.random.default_rng(3)
    x = _tensor(_inputs(rng, n, 144, torch.float32))
    g = _tensor(_inputs(rng, n, 144, torch.float32))
    a = [P.norm_forward(fields, x) for _ in range(2)]
    b = [P.norm_backward(fields, x, g) for _ in range(2)]
    assert torch.equal(a[0], a[1]) and torch.equal(b[0], b[1])


def test_norm_pool_argument_errors():
    fields = ((0, 2),)
    x = torch.zeros((4, 2), device=DEV)
    with pytest.raises(_abi.SSConvError) as e:
        P.norm_forward(fields, x, eps=0.0)
    assert e.value.code == _abi.E_INVALID
    with pytest.raises(_abi.SSConvError) as e:
        P.norm_forward(((0, 1025),), torch.zeros((2, 1025), device=DEV))
    assert e.value.code == _abi.E_INVALID
    P.norm_forward(fields, torch.zeros((0, 2), device=DEV))          # n = 0: no-op
    coords = _tensor(np.array([[0, 1, 1, 1], [0, 2, 2, 2]], np.int32))
    rb3 = P.Rulebook(coords, 4, 3, 1, True)
    with pytest.raises(_abi.SSConvError) as e:
        P.pool_forward(torch.zeros((2, 4), device=DEV), rb3)         # not a pooling rule book
    assert e.value.code == _abi.E_INVALID
    rb2 = P.Rulebook(coords, 4, 2, 2, False)
    W = torch.zeros((8, 4, 4), device=DEV)
    with pytest.raises(_abi.SSConvError) as e:
        P.forward(torch.zeros((2, 4), device=DEV), rb2, W)           # pooling windows are not a conv kernel
    assert e.value.code == _abi.E_INVALID
    for ks, st, sub in [(2, 1, False), (2, 1, True), (4, 2, False)]:
        with pytest.raises(_abi.SSConvError) as e:
            P.Rulebook(coords, 4, ks, st, sub)
        assert e.value.code == _abi.E_INVALID
    rb3.close()
    rb2.close()


# ---- the downsampling block ---------------------------------------------------------------

def test_block_forward_backward_matches_oracle():
    """SS-Conv -> Norm -> gate -> pooling on the 32 objects of the block workload, through the
    C ABI, against the composed fp64 oracle."""
    i = 6
    spec = CONFIGS[i]
    L = layers_of(i)[0]
    print(f"block n={len(L.coords_in)}", flush=True)
    pc, want, g, d_in, dw = block_reference(i)
    blk = DownBlock.create(L.spec, L.coeffs, spec.grid, DEV)
    oc_, out = blk.forward(_tensor(L.coords_in), _tensor(features_of(i)))
    np.testing.assert_array_equal(oc_.cpu().numpy(), pc)
    e0 = rel_err(out.cpu().numpy(), want)
    gf, gc = blk.backward(_tensor(g.astype(np.float32)))
    e1, e2 = rel_err(gf.cpu().numpy(), d_in), rel_err(gc.cpu().numpy(), dw)
    print(f"block errors out {e0:.3e} grad_feats {e1:.3e} grad_coeffs {e2:.3e}", flush=True)
    assert max(e0, e1, e2) < 1e-4
    blk.close()

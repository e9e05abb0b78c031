"""GPU parity: the HIP library against the fp64 oracle on the five seeded workloads.

Rule books and hash tables must match exactly (same sets, same order); fp32
features within 1e-4 and bf16 within 2e-2, as L_inf error over the L_inf norm
of the oracle result.  Every call goes through the C ABI.
"""
import numpy as np
import pytest

from cases import coords_of, features_of, layers_of, rel_err, single_layer_reference
from workloads import CONFIGS

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
P = pytest.importorskip("paper_2111_07383_amd")

DEV = "cuda:0"
TOL = {"f32": 1e-4, "bf16": 2e-2}


def _dt(i):
    return torch.bfloat16 if CONFIGS[i].dtype == "bf16" else torch.float32


def _tensor(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
    return t.to(dtype) if dtype is not None else t


def _pair_keys(s, o, i):
    return (np.asarray(s, np.int64) << 42) | (np.asarray(o, np.int64) << 21) | np.asarray(i, np.int64)


def _check_rulebook(L, rb):
    K = L.spec.ksize ** 3
    assert rb.n_in == len(L.coords_in) and rb.n_out == len(L.coords_out)
    np.testing.assert_array_equal(rb.out_coords().cpu().numpy(), L.coords_out)
    counts = np.array([len(r) for r in L.R])
    np.testing.assert_array_equal(rb.pair_counts, counts)
    got = rb.pairs().cpu().numpy().astype(np.int64)
    want = np.concatenate([r for r in L.R if len(r)] or [np.zeros((0, 2), np.int64)])
    s_idx = np.repeat(np.arange(K), counts)
    # same set of (s, out, in) triples, and the same order (grouped by s, out rows ascending)
    assert np.array_equal(np.sort(_pair_keys(s_idx, got[:, 0], got[:, 1])), np.sort(_pair_keys(s_idx, want[:, 0], want[:, 1])))
    np.testing.assert_array_equal(got, want)
    np.testing.assert_array_equal(rb.neighbours().cpu().numpy(), L.nbr)


def _check_hash(coords, grid, slots):
    slots = slots.cpu().numpy().view(np.uint64)
    occ = slots != np.uint64(0xFFFFFFFFFFFFFFFF)
    keys = (slots[occ] >> np.uint64(32)).astype(np.int64)
    rows = (slots[occ] & np.uint64(0xFFFFFFFF)).astype(np.int64)
    c = coords.astype(np.int64)
    want = ((c[:, 0] * grid + c[:, 1]) * grid + c[:, 2]) * grid + c[:, 3]
    got = np.zeros(len(c), np.int64) - 1
    assert len(rows) == len(c) and len(np.unique(rows)) == len(c)
    got[rows] = keys
    np.testing.assert_array_equal(got, want)


@pytest.mark.parametrize("i", [1, 2, 3, 4, 5])
def test_rulebook_and_hash_exact(i):
    spec = CONFIGS[i]
    for L in layers_of(i):
        print(f"rulebook config {i} grid {L.grid} k{L.spec.ksize} s{L.spec.stride} n={len(L.coords_in)}", flush=True)
        rb = P.Rulebook(_tensor(L.coords_in), L.grid, L.spec.ksize, L.spec.stride, L.spec.submanifold)
        _check_rulebook(L, rb)
        _check_hash(L.coords_in, L.grid, rb.hash_slots(0))
        if not L.spec.submanifold:
            _check_hash(L.coords_out, -(-L.grid // L.spec.stride), rb.hash_slots(1))
        rb.close()


@pytest.mark.parametrize("i", [1, 2, 3, 4, 5])
def test_synth_matches_oracle(i):
    spec = CONFIGS[i]
    for L in layers_of(i):
        desc = P.layer_desc(L.spec)
        basis = _tensor(P.basis_build(desc))
        W = P.synth_kernel(desc, basis, _tensor(L.coeffs), torch.float32).cpu().numpy()
        kap = L.lay.kappa(L.coeffs)                      # fp64, unrounded
        assert rel_err(W, kap) < 1e-6
        if spec.dtype == "bf16":
            Wb = P.synth_kernel(desc, basis, _tensor(L.coeffs), torch.bfloat16).float().cpu().numpy()
            assert rel_err(Wb, L.kappa) < 2e-2
            assert np.abs(Wb - L.kappa).max() <= 2.0 ** -8 * np.abs(L.kappa).max()


def _layer_io(i):
    L = layers_of(i)[0]
    dt = _dt(i)
    desc = P.layer_desc(L.spec)
    basis = _tensor(P.basis_build(desc))
    coeffs = _tensor(L.coeffs)
    rb = P.Rulebook(_tensor(L.coords_in), L.grid, L.spec.ksize, L.spec.stride, L.spec.submanifold)
    W = P.synth_kernel(desc, basis, coeffs, dt)
    feats = _tensor(features_of(i), dt)
    return L, dt, desc, basis, rb, W, feats


@pytest.mark.parametrize("i", [1, 2, 3, 4, 6])
def test_forward_matches_oracle(i):
    print(f"forward config {i}", flush=True)
    L, dt, desc, basis, rb, W, feats = _layer_io(i)
    out = P.forward(feats, rb, W).float().cpu().numpy()
    want, *_ = single_layer_reference(i)
    err = rel_err(out, want)
    print(f"config {i} forward rel err {err:.3e}", flush=True)
    assert err < TOL[CONFIGS[i].dtype]
    rb.close()


@pytest.mark.parametrize("i", [1, 2, 3, 4, 6])
def test_backward_matches_oracle(i):
    print(f"backward config {i}", flush=True)
    L, dt, desc, basis, rb, W, feats = _layer_io(i)
    _, g, d_in, dw = single_layer_reference(i)
    gf, gc = P.backward(feats, _tensor(g, dt), rb, W, desc, basis)
    e1, e2 = rel_err(gf.float().cpu().numpy(), d_in), rel_err(gc.cpu().numpy(), dw)
    print(f"config {i} grad_feats rel err {e1:.3e} grad_coeffs rel err {e2:.3e}", flush=True)
    tol = TOL[CONFIGS[i].dtype]
    assert e1 < tol and e2 < tol
    rb.close()


def test_bf16_diagnostic_against_unrounded_inputs():
    """Diagnostic second reference of the bf16 workload: the fp64 oracle on the fp32 features and
    kernel before their rounding to bfloat16.  The gate stays the reference on the rounded inputs
    (what the GPU is given); this one also contains the input quantisation.  Each rounded operand
    is within 2^-9 of its value (relative), so a product is within about 2^-8, and the sum of
    ~20 * 208 such products with random signs stays within a few 2^-8 of the L_inf norm."""
    from workloads.gen import make_features
    i = 4
    L, dt, desc, basis, rb, W, feats = _layer_io(i)
    out = P.forward(feats, rb, W).float().cpu().numpy()
    rb.close()
    want_rounded, *_ = single_layer_reference(i)
    f32 = make_features(CONFIGS[i], len(L.coords_in), L.spec.cin, rounded=False).astype(np.float64)
    kap = L.lay.kappa(L.coeffs, bf16=False)
    from oracle import conv as oc
    want_unrounded = oc.forward(f32, L.R, kap, len(L.coords_out))
    e_gate, e_diag = rel_err(out, want_rounded), rel_err(out, want_unrounded)
    e_inputs = rel_err(want_rounded, want_unrounded)
    print(f"config 4 forward: vs rounded inputs {e_gate:.3e}, vs unrounded inputs {e_diag:.3e} "
          f"(oracle rounded vs unrounded {e_inputs:.3e})", flush=True)
    assert e_gate < TOL["bf16"]
    assert e_diag < 4 * 2.0 ** -8


_KGRAD_LAYERS = {
    "c4": None,                                                     # the 128^3 scene layer, tile 224
    "w2": (((0, 16), (1, 8)), ((0, 16), (1, 8), (2, 4))),           # 40 -> 60: tile 64
    "w4": (((0, 16), (1, 8), (2, 4), (1, 8), (0, 16)), ((0, 32), (1, 16), (2, 8))),  # 100 -> 120: tile 128
    "w7x2": (((0, 32), (1, 32), (2, 16)), ((0, 32), (1, 32), (2, 16), (1, 12), (0, 56))),  # 208 -> 300: 2 tiles
}


@pytest.mark.parametrize("name", list(_KGRAD_LAYERS))
def test_bf16_kernel_gradient_staging_layouts_bit_identical(name):
    """The bf16 kernel gradient with its operands staged in 64-byte quads (default) against the
    16-byte column layout (override 12): the MFMAs read the same operands, so the coefficient
    gradient agrees bit for bit.  Tiles of 64, 128 and 224 channels, one layer with two output
    tiles, ragged channel counts inside the tiles."""
    from workloads.configs import LayerSpec
    print(f"bf16 kernel gradient staging, {name}", flush=True)
    if name == "c4":
        L, dt, desc, basis, rb, W, feats = _layer_io(4)
        spec = L.spec
    else:
        fin, fout = _KGRAD_LAYERS[name]
        spec = LayerSpec(3, 1, True, fin, fout, shells=(0.0, 1.0))
        L6 = layers_of(6)[0]
        rb = P.Rulebook(_tensor(L6.coords_in), L6.grid, 3, 1, True)
        desc = P.layer_desc(spec)
        basis = _tensor(P.basis_build(desc))
        gen = torch.Generator(DEV).manual_seed(len(name))
        coeffs = torch.randn(P.basis_info(desc)[1], device=DEV, generator=gen)
        W = P.synth_kernel(desc, basis, coeffs, torch.bfloat16)
        feats = torch.randn(rb.n_in, spec.cin, device=DEV, generator=gen).to(torch.bfloat16)
    g = torch.randn(rb.n_out, spec.cout, device=DEV, generator=torch.Generator(DEV).manual_seed(7)).to(torch.bfloat16)
    got = []
    for variant in (0, 12):
        P.debug_set(3, variant)
        try:
            got.append(P.backward(feats, g, rb, W, desc, basis, need_feats=False)[1])
        finally:
            P.debug_set(3, 0)
    assert torch.equal(got[0], got[1])
    rb.close()


def test_forward_backward_deterministic():
    L, dt, desc, basis, rb, W, feats = _layer_io(2)
    g = torch.randn(rb.n_out, L.spec.cout, device=DEV, generator=torch.Generator(DEV).manual_seed(0))
    o1 = P.forward(feats, rb, W)
    o2 = P.forward(feats, rb, W)
    a1, b1 = P.backward(feats, g, rb, W, desc, basis)
    a2, b2 = P.backward(feats, g, rb, W, desc, basis)
    assert torch.equal(o1, o2) and torch.equal(a1, a2) and torch.equal(b1, b2)
    rb2 = P.Rulebook(_tensor(L.coords_in), L.grid, L.spec.ksize, 1, True)
    assert torch.equal(rb2.pairs(), rb.pairs())
    rb.close()
    rb2.close()


@pytest.mark.parametrize("i,variant", [(2, 1), (2, 2), (2, 3), (3, 3), (2, 7), (3, 7), (4, 5), (4, 6), (2, 8),
                                       (3, 8), (1, 9), (2, 9), (3, 10), (6, 10)])
def test_kernel_selection_overrides(i, variant):
    """Every alternative kernel configuration (forced from the host) stays within tolerance."""
    print(f"config {i} kernel variant {variant}", flush=True)
    L, dt, desc, basis, rb, W, feats = _layer_io(i)
    want, g, d_in, dw = single_layer_reference(i)
    P.debug_set(3, variant)
    try:
        out = P.forward(feats, rb, W).float().cpu().numpy()
        gf, gc = P.backward(feats, _tensor(g, dt), rb, W, desc, basis)
    finally:
        P.debug_set(3, 0)
    tol = TOL[CONFIGS[i].dtype]
    errs = rel_err(out, want), rel_err(gf.float().cpu().numpy(), d_in), rel_err(gc.cpu().numpy(), dw)
    print(f"config {i} variant {variant} errors {errs}", flush=True)
    assert max(errs) < tol
    rb.close()


def test_pair_path_deterministic():
    """The sparse stride-2 layer runs on the pair-list path: same bits on every call."""
    L, dt, desc, basis, rb, W, feats = _layer_io(3)
    g = torch.randn(rb.n_out, L.spec.cout, device=DEV, generator=torch.Generator(DEV).manual_seed(1))
    o1, o2 = P.forward(feats, rb, W), P.forward(feats, rb, W)
    a1, _ = P.backward(feats, g, rb, W, desc, basis, need_coeffs=False)
    a2, _ = P.backward(feats, g, rb, W, desc, basis, need_coeffs=False)
    assert torch.equal(o1, o2) and torch.equal(a1, a2)
    rb.close()


@pytest.mark.parametrize("i", [3, 2])
def test_backward_fork_bit_identical(i):
    """The coefficient gradient forked onto the library's second stream gives the same bits as on
    the caller's stream (override 11): all of it next to a pair-list feature gradient (workload 3),
    its reduction and synthesis adjoint next to the fp32 gather kernel (workload 2)."""
    L, dt, desc, basis, rb, W, feats = _layer_io(i)
    g = torch.randn(rb.n_out, L.spec.cout, device=DEV, generator=torch.Generator(DEV).manual_seed(2)).to(dt)
    a1, b1 = P.backward(feats, g, rb, W, desc, basis)
    P.debug_set(3, 11)
    try:
        a2, b2 = P.backward(feats, g, rb, W, desc, basis)
    finally:
        P.debug_set(3, 0)
    assert torch.equal(a1, a2) and torch.equal(b1, b2)
    rb.close()

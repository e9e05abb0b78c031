"""GPU edge cases and failure paths of the C ABI.

Failures are forced from the host (bad arguments, duplicate or out-of-grid
sites, a forced small hash capacity, a forced allocation failure); every
kernel still runs to completion.  Ragged shapes exercise partial tiles, odd
channel counts (scalar gather path) and empty inputs.
"""
import numpy as np
import pytest

from cases import rel_err
from oracle import conv as oc
from oracle import rulebook as orb
from workloads.configs import LayerSpec

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
P = pytest.importorskip("paper_2111_07383_amd")
from paper_2111_07383_amd._abi import E_BOUNDS, E_DUPLICATE, E_HASH_FULL, E_INVALID, E_NOMEM, SSConvError  # noqa: E402

DEV = "cuda:0"


def _coords(seed, n, grid, batch=1):
    rng = np.random.default_rng(seed)
    c = np.concatenate([rng.integers(0, batch, (n, 1)), rng.integers(0, grid, (n, 3))], 1)
    return np.unique(c, axis=0).astype(np.int32)


def _code(fn):
    with pytest.raises(SSConvError) as e:
        fn()
    return e.value.code


def test_error_codes():
    c = torch.from_numpy(_coords(0, 50, 8)).to(DEV)
    dup = torch.cat([c, c[:1]])
    assert _code(lambda: P.Rulebook(dup, 8, 3)) == E_DUPLICATE
    # generated output sets (stride 2, 2x2x2 pooling windows) stop before writing any map entry
    assert _code(lambda: P.Rulebook(dup, 8, 3, 2, False)) == E_DUPLICATE
    assert _code(lambda: P.Rulebook(dup, 8, 2, 2, False)) == E_DUPLICATE
    bad = c.clone()
    bad[3, 2] = 8
    assert _code(lambda: P.Rulebook(bad, 8, 3)) == E_BOUNDS
    neg = c.clone()
    neg[0, 0] = -1
    assert _code(lambda: P.Rulebook(neg, 8, 3)) == E_BOUNDS
    assert _code(lambda: P.Rulebook(c, 8, 3, stride=2, submanifold=True)) == E_INVALID
    assert _code(lambda: P.Rulebook(c, 8, 4)) == E_INVALID
    assert _code(lambda: P.Rulebook(c, 8, 3, stride=3, submanifold=False)) == E_INVALID
    big = c.clone()
    big[:, 0] = 9_000_000                               # (b+1) * 8^3 exceeds 2^32
    assert _code(lambda: P.Rulebook(big, 8, 3)) == E_BOUNDS
    P.debug_set(1, 16)                                  # 16 slots for 50 sites
    try:
        assert _code(lambda: P.Rulebook(c, 8, 3)) == E_HASH_FULL
        assert _code(lambda: P.Rulebook(c, 8, 3, stride=2, submanifold=False)) == E_HASH_FULL
    finally:
        P.debug_set(1, 0)
    P.debug_set(2, 1)                                   # a submanifold build's one allocation fails
    assert _code(lambda: P.Rulebook(c, 8, 3)) == E_NOMEM
    P.debug_set(2, 2)                                   # a stride-2 build's second allocation fails
    assert _code(lambda: P.Rulebook(c, 8, 3, stride=2, submanifold=False)) == E_NOMEM
    P.debug_set(2, 0)
    rb = P.Rulebook(c, 8, 3)                            # library still healthy
    assert rb.n_out == len(c)
    rb.close()


def test_async_rulebook_matches_sync():
    """ssconv_build_rulebook_async: pairs, neighbour map and hash contents equal the synchronous
    build's; a
    bf16 forward queued before the build is settled, the fp32 forward (which settles it) and the
    backward give the same bits as on the synchronous build."""
    from cases import coords_of, layers_of
    L = layers_of(4)[0]
    c = torch.from_numpy(L.coords_in).to(DEV)
    gen = torch.Generator(DEV).manual_seed(3)
    rb_s = P.Rulebook(c, L.grid, 3, 1, True)
    rb_a = P.Rulebook(c, L.grid, 3, 1, True, asynchronous=True)
    W = (torch.randn(27, 16, 24, device=DEV, generator=gen) * 0.2).to(torch.bfloat16)
    f = torch.randn(rb_s.n_in, 24, device=DEV, generator=gen).to(torch.bfloat16)
    y_a = P.forward(f, rb_a, W)                         # queued on the unsettled build
    y_s = P.forward(f, rb_s, W)
    assert torch.equal(y_a, y_s)
    assert rb_a.n_pairs == rb_s.n_pairs and np.array_equal(rb_a.pair_counts, rb_s.pair_counts)
    assert torch.equal(rb_a.pairs(), rb_s.pairs()) and torch.equal(rb_a.neighbours(), rb_s.neighbours())
    # the table's contents as a set (concurrent inserts place keys in race-dependent slots)
    assert torch.equal(torch.sort(rb_a.hash_slots(0))[0], torch.sort(rb_s.hash_slots(0))[0])
    g = torch.randn(rb_s.n_out, 16, device=DEV, generator=gen).to(torch.bfloat16)
    assert torch.equal(P.backward(f, g, rb_a, W, need_coeffs=False)[0], P.backward(f, g, rb_s, W, need_coeffs=False)[0])
    rb_a.close()
    rb_a = P.Rulebook(c, L.grid, 3, 1, True, asynchronous=True)
    W32, f32 = W.float(), f.float()
    assert torch.equal(P.forward(f32, rb_a, W32), P.forward(f32, rb_s, W32))   # fp32 settles first
    rb_a.close()
    rb_s.close()
    P.Rulebook(c, L.grid, 3, 1, True, asynchronous=True).close()   # destroyed before it is settled


def test_async_rulebook_reports_errors_when_settled():
    """The errors the device detects surface when the asynchronous build is settled: by wait(),
    the pair counts, an fp32 forward or the backward; a bf16 forward queued before that runs (its
    result is undefined) without any access outside the buffers."""
    c = torch.from_numpy(_coords(0, 50, 8)).to(DEV)
    dup = torch.cat([c, c[:1]])
    rb = P.Rulebook(dup, 8, 3, asynchronous=True)       # no error yet
    gen = torch.Generator(DEV).manual_seed(4)
    W = torch.randn(27, 8, 8, device=DEV, generator=gen).to(torch.bfloat16)
    f = torch.randn(len(dup), 8, device=DEV, generator=gen).to(torch.bfloat16)
    P.forward(f, rb, W)
    torch.cuda.synchronize()
    assert _code(lambda: rb.wait()) == E_DUPLICATE
    assert _code(lambda: rb.wait()) == E_DUPLICATE      # the same result on every call
    assert _code(lambda: rb.n_pairs) == E_DUPLICATE
    assert _code(lambda: P.forward(f.float(), rb, W.float())) == E_DUPLICATE
    g = torch.zeros(len(dup), 8, device=DEV, dtype=torch.bfloat16)
    assert _code(lambda: P.backward(f, g, rb, W, need_coeffs=False)) == E_DUPLICATE
    rb.close()
    P.debug_set(1, 16)                                  # 16 slots for 50 sites
    try:
        rb = P.Rulebook(c, 8, 3, asynchronous=True)
        assert _code(lambda: rb.wait()) == E_HASH_FULL
        rb.close()
    finally:
        P.debug_set(1, 0)
    rb = P.Rulebook(c, 8, 3, asynchronous=True)         # a clean build settles without error
    rb.wait()
    assert rb.n_pairs > 0
    rb.close()


def test_empty_input():
    c = torch.zeros((0, 4), dtype=torch.int32, device=DEV)
    for stride, sub in ((1, True), (2, False)):
        rb = P.Rulebook(c, 16, 3, stride, sub)
        assert rb.n_in == 0 and rb.n_out == 0 and rb.n_pairs == 0
        W = torch.zeros((27, 8, 4), device=DEV)
        out = P.forward(torch.zeros((0, 4), device=DEV), rb, W)
        assert out.shape == (0, 8)
        rb.close()


@pytest.mark.parametrize("ksize,stride,sub,dtype", [
    (3, 1, True, "f32"), (5, 1, True, "f32"), (3, 2, False, "f32"), (3, 1, False, "f32"),
    (5, 2, False, "f32"), (1, 1, True, "f32"), (3, 1, True, "bf16"), (5, 2, False, "bf16")])
def test_ragged_layers(ksize, stride, sub, dtype):
    """Odd channel counts (13 -> 14), a partial last tile and several batch entries."""
    spec = LayerSpec(ksize, stride, sub, ((0, 2), (1, 2), (2, 1)), ((0, 1), (1, 1), (2, 2)),
                     shells=tuple(float(m) for m in range(ksize // 2 + 1)))
    grid = 12
    c = _coords(ksize * 7 + stride, 333, grid, batch=3)
    lay = oc.Layer(spec)
    rng = np.random.default_rng(5)
    w = rng.standard_normal(lay.n_coeff).astype(np.float32)
    f = rng.standard_normal((len(c), spec.cin)).astype(np.float32)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    if dtype == "bf16":
        f = torch.from_numpy(f).to(tdt).float().numpy()
    co = orb.output_sites(c, grid, ksize, stride, sub)
    R = orb.rulebook(c, co, ksize, stride)
    kap = lay.kappa(w, bf16=(dtype == "bf16"))
    want = oc.forward(f, R, kap, len(co))
    g = rng.standard_normal((len(co), spec.cout)).astype(np.float32)
    if dtype == "bf16":
        g = torch.from_numpy(g).to(tdt).float().numpy()
    d_in = oc.grad_feats(g, R, kap, len(c))
    dw = oc.synth_adjoint(spec, lay.basis, oc.grad_kappa(f, g, R, kap.shape))

    desc = P.layer_desc(spec)
    basis = torch.from_numpy(P.basis_build(desc)).to(DEV)
    rb = P.Rulebook(torch.from_numpy(c).to(DEV), grid, ksize, stride, sub)
    np.testing.assert_array_equal(rb.out_coords().cpu().numpy(), co)
    W = P.synth_kernel(desc, basis, torch.from_numpy(w).to(DEV), tdt)
    ft = torch.from_numpy(f).to(DEV).to(tdt)
    out = P.forward(ft, rb, W).float().cpu().numpy()
    gf, gc = P.backward(ft, torch.from_numpy(g).to(DEV).to(tdt), rb, W, desc, basis)
    tol = 2e-2 if dtype == "bf16" else 1e-4
    assert rel_err(out, want) < tol
    assert rel_err(gf.float().cpu().numpy(), d_in) < tol
    assert rel_err(gc.cpu().numpy(), dw) < tol
    rb.close()


def test_row_order_independence():
    """Permuting the input rows permutes submanifold outputs the same way."""
    spec = LayerSpec(3, 1, True, ((0, 4), (1, 4)), ((0, 4), (1, 4)), shells=(0.0, 1.0))
    c = _coords(11, 2000, 20, batch=2)
    perm = np.random.default_rng(1).permutation(len(c))
    lay = oc.Layer(spec)
    rng = np.random.default_rng(2)
    w = torch.from_numpy(rng.standard_normal(lay.n_coeff).astype(np.float32)).to(DEV)
    f = rng.standard_normal((len(c), spec.cin)).astype(np.float32)
    desc = P.layer_desc(spec)
    basis = torch.from_numpy(P.basis_build(desc)).to(DEV)
    W = P.synth_kernel(desc, basis, w)
    outs = []
    for cc, ff in ((c, f), (c[perm], f[perm])):
        rb = P.Rulebook(torch.from_numpy(np.ascontiguousarray(cc)).to(DEV), 20, 3)
        outs.append(P.forward(torch.from_numpy(np.ascontiguousarray(ff)).to(DEV), rb, W).cpu().numpy())
        rb.close()
    assert rel_err(outs[1], outs[0][perm]) < 1e-6


@pytest.mark.parametrize("dt", [torch.float32, torch.bfloat16])
def test_kernel_timing_hook(dt):
    c = torch.from_numpy(_coords(5, 3000, 24)).to(DEV)
    rb = P.Rulebook(c, 24, 3)
    W = (torch.randn((27, 48, 32), device=DEV) * 0.1).to(dt)
    x = torch.randn((rb.n_in, 32), device=DEV).to(dt)
    P.debug_set(4, 1)
    try:
        y0 = P.forward(x, rb, W)
        y1 = P.forward(x, rb, W)
        n, ms = P.debug_kernel_ms()
        assert n == 2 and ms > 0.0
        torch.testing.assert_close(y0, y1, rtol=0, atol=0)
        P.debug_set(4, 1)                                # switching on again clears the log
        assert _code(P.debug_kernel_ms) == E_INVALID
    finally:
        P.debug_set(4, 0)
    P.forward(x, rb, W)                                  # timing off: nothing recorded
    assert _code(P.debug_kernel_ms) == E_INVALID
    rb.close()


def test_device_memory_cache():
    """Freed library blocks are cached and reused, also on another stream (after an event wait),
    without changing any result; empty_cache releases them."""
    P.empty_cache()
    assert P.cached_bytes() == 0
    c = torch.from_numpy(_coords(11, 4000, 24)).to(DEV)
    ref = P.Rulebook(c, 24, 3)
    W = (torch.randn((27, 48, 32), device=DEV) * 0.1).to(torch.bfloat16)
    x = torch.randn((ref.n_in, 32), device=DEV).to(torch.bfloat16)
    y_ref = P.forward(x, ref, W)
    P.Rulebook(c, 24, 3).close()
    assert P.cached_bytes() > 0
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for _ in range(2):                               # blocks freed on the default stream, reused here
            rb = P.Rulebook(c, 24, 3, stream=side)
            y = P.forward(x, rb, W, stream=side)
            nb, pairs = rb.neighbours(stream=side), rb.pairs(stream=side)
            side.synchronize()
            torch.testing.assert_close(nb, ref.neighbours(), rtol=0, atol=0)
            torch.testing.assert_close(pairs, ref.pairs(), rtol=0, atol=0)
            torch.testing.assert_close(y, y_ref, rtol=0, atol=0)
            rb.close()
    torch.cuda.synchronize()
    P.empty_cache()
    assert P.cached_bytes() == 0
    rb = P.Rulebook(c, 24, 3)                            # allocations after emptying still work
    torch.testing.assert_close(rb.neighbours(), ref.neighbours(), rtol=0, atol=0)
    rb.close()
    ref.close()


@pytest.mark.parametrize("ksize,stride,sub", [(3, 1, True), (5, 1, True), (3, 2, False), (1, 1, True)])
@pytest.mark.parametrize("fields_out", [((0, 4), (1, 3), (2, 1)), ((0, 4), (1, 2), (2, 2))])
def test_pair_path_ragged(ksize, stride, sub, fields_out):
    """The pair-list path forced on small layers: 12 input channels; 18 outputs (a partial column
    block and the scalar per-row sum) or 20 (both directions on the pair path), several batch
    entries, against the oracle."""
    spec = LayerSpec(ksize, stride, sub, ((0, 4), (1, 1), (2, 1)), fields_out,
                     shells=tuple(float(m) for m in range(ksize // 2 + 1)))
    grid = 12
    c = _coords(ksize * 11 + stride, 400, grid, batch=3)
    lay = oc.Layer(spec)
    rng = np.random.default_rng(ksize + spec.cout)
    w = rng.standard_normal(lay.n_coeff).astype(np.float32)
    f = rng.standard_normal((len(c), spec.cin)).astype(np.float32)
    co = orb.output_sites(c, grid, ksize, stride, sub)
    R = orb.rulebook(c, co, ksize, stride)
    kap = lay.kappa(w)
    g = rng.standard_normal((len(co), spec.cout)).astype(np.float32)
    want = oc.forward(f, R, kap, len(co))
    d_in = oc.grad_feats(g, R, kap, len(c))
    dw = oc.synth_adjoint(spec, lay.basis, oc.grad_kappa(f, g, R, kap.shape))
    desc = P.layer_desc(spec)
    basis = torch.from_numpy(P.basis_build(desc)).to(DEV)
    rb = P.Rulebook(torch.from_numpy(c).to(DEV), grid, ksize, stride, sub)
    W = P.synth_kernel(desc, basis, torch.from_numpy(w).to(DEV))
    ft = torch.from_numpy(f).to(DEV)
    P.debug_set(3, 9)
    try:
        out = P.forward(ft, rb, W).cpu().numpy()
        gf, gc = P.backward(ft, torch.from_numpy(g).to(DEV), rb, W, desc, basis)
    finally:
        P.debug_set(3, 0)
    errs = rel_err(out, want), rel_err(gf.cpu().numpy(), d_in), rel_err(gc.cpu().numpy(), dw)
    print(f"pair path k{ksize} s{stride} cout {spec.cout}: {errs}", flush=True)
    assert max(errs) < 1e-4
    rb.close()


@pytest.mark.parametrize("ksize,stride", [(3, 2), (3, 1)])
def test_generated_output_table_on_request(ksize, stride):
    """A generated output set's coordinate table is filled only when asked for: the rule book
    built without it matches the oracle's pairs, and the table, read twice, holds exactly the
    output sites with their rows."""
    grid = 19
    c = _coords(21, 1500, grid, batch=3)
    rb = P.Rulebook(torch.from_numpy(c).to(DEV), grid, ksize, stride, False)
    try:
        oc_out = rb.out_coords().cpu().numpy()
        ref = orb.rulebook(c, oc_out, ksize, stride)
        got = rb.pairs().cpu().numpy()
        counts = [len(r) for r in ref]
        off = np.concatenate([[0], np.cumsum(counts)])
        assert got.shape[0] == off[-1]
        for s, r in enumerate(ref):
            assert np.array_equal(got[off[s]:off[s + 1]], np.asarray(r, dtype=np.int32).reshape(-1, 2))
        t1 = rb.hash_slots(1).cpu().numpy().view(np.uint64)
        t2 = rb.hash_slots(1).cpu().numpy().view(np.uint64)
        assert np.array_equal(t1, t2)
        full = t1[t1 != np.uint64(0xFFFFFFFFFFFFFFFF)]
        go = -(-grid // stride)
        b, x, y, z = (oc_out[:, i].astype(np.uint64) for i in range(4))
        keys = ((b * go + x) * go + y) * go + z
        want = np.sort((keys << np.uint64(32)) | np.arange(len(oc_out), dtype=np.uint64))
        assert np.array_equal(np.sort(full), want)
    finally:
        rb.close()

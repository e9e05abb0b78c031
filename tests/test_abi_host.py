"""CPU checks of the C ABI library: it loads, exports every declared symbol, and its
host-only basis builder (Racah Clebsch-Gordan route) agrees with the oracle's
null-space basis.  No GPU call is made here.
"""
import os
import re

import numpy as np
import pytest

from oracle import basis as ob
from oracle.conv import Layer
from workloads import CONFIGS
from workloads.configs import LayerSpec

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ssconv.h")


@pytest.fixture(scope="module")
def abi():
    from paper_2111_07383_amd import _abi
    if not os.path.exists(_abi.LIB_PATH):
        pytest.skip("libssconv.so not built")
    return _abi


def declared_symbols():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(ssconv_[a-z_0-9]+)\s*\(", text)))


def test_library_exports_every_declared_symbol(abi):
    import ctypes
    lib = ctypes.CDLL(abi.LIB_PATH)
    names = declared_symbols()
    assert len(names) >= 18
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(abi.SIGNATURES), "binding and header disagree"


def _oracle_flat(spec):
    lay = Layer(spec)
    ks = sorted({l for l, _ in spec.fields_out})
    ls = sorted({l for l, _ in spec.fields_in})
    return lay, np.concatenate([lay.basis[(k, l)].reshape(-1) for k in ks for l in ls])


EXTRA = [
    LayerSpec(1, 1, True, ((0, 2), (1, 1), (2, 1)), ((0, 1), (1, 2), (2, 1)), shells=(0.0,)),
    LayerSpec(5, 1, True, ((1, 1), (2, 1)), ((2, 1), (1, 1)), shells=(0.0, 1.0, 2.0), jmax=1),
    LayerSpec(3, 1, True, ((0, 1), (1, 1), (2, 1)), ((0, 1), (1, 1), (2, 1)), shells=(0.0, 1.0), eps=0.35),
]


@pytest.mark.parametrize("spec", [L for i in range(1, 6) for L in CONFIGS[i].layers] + EXTRA)
def test_host_basis_matches_oracle(abi, spec):
    from paper_2111_07383_amd import binding as B
    d = B.layer_desc(spec)
    floats, ncoef = B.basis_info(d)
    lay, want = _oracle_flat(spec)
    assert ncoef == lay.n_coeff == ob.coeff_count(spec)
    assert floats == want.size
    got = B.basis_build(d)
    assert np.abs(got - want).max() < 1e-7          # fp32 rounding of a unit-norm basis


def test_invalid_descriptors(abi):
    from paper_2111_07383_amd import binding as B
    bad = B.basis_desc(((0, 1),), ((0, 1),), 4, (0.0,))
    with pytest.raises(abi.SSConvError) as e:
        B.basis_info(bad)
    assert e.value.code == abi.E_INVALID
    bad = B.basis_desc(((5, 1),), ((0, 1),), 3, (0.0,))
    with pytest.raises(abi.SSConvError):
        B.basis_info(bad)
    with pytest.raises(abi.SSConvError):
        B.debug_set(9, 1)


def test_kernel_timing_without_timed_call(abi):
    from paper_2111_07383_amd import binding as B
    B.debug_set(4, 0)
    with pytest.raises(abi.SSConvError) as e:       # nothing timed on this thread: no device call made
        B.debug_kernel_ms()
    assert e.value.code == abi.E_INVALID


def test_wigner_d_matches_oracle(abi):
    """The library's Wigner-D (projection by an exact sphere quadrature) against the oracle's
    (least squares over random directions) for random rotations and every order up to 4."""
    from oracle import sh
    from paper_2111_07383_amd.binding import wigner_d
    rng = np.random.default_rng(11)
    for k in range(6):
        q = rng.standard_normal(4)
        q /= np.linalg.norm(q)
        w, x, y, z = q
        R = np.array([[1 - 2 * (y * y + z * z), 2 * (x * y - z * w), 2 * (x * z + y * w)],
                      [2 * (x * y + z * w), 1 - 2 * (x * x + z * z), 2 * (y * z - x * w)],
                      [2 * (x * z - y * w), 2 * (y * z + x * w), 1 - 2 * (x * x + y * y)]])
        for l in range(5):
            np.testing.assert_allclose(wigner_d(l, R), sh.wigner_d(l, R), atol=1e-12)

"""Pins for two oracle parts that every other pin takes for granted.

* ``conv.round_bf16``: the rounding of fp32 values to bfloat16 that the bf16
  workload applies to its features and to the synthesised kernel (the oracle
  then computes in fp64 from exactly the values the GPU sees).  Pinned against
  literal round-to-nearest-even cases worked out by hand on the bit patterns,
  and against PyTorch's own CPU float32 -> bfloat16 conversion (an independent
  implementation) on a million random values spread over every exponent.
* ``basis.radial``: the Gaussian radial profile phi^m(r) = exp(-(r - m)^2 /
  (2 eps^2)) of Sec. 3.2.1, Eq. 8 (eps = 0.6 as in the Plain12 setting of
  Sec. 5.1).  Pinned by literal values of the closed form (computed with
  Python's ``decimal`` module at 30 digits, not with the oracle), both
  directly and through a whole layer: for scalar fields the steerable kernel is
  an isotropic stencil whose value at offset s is proportional to phi^m(|s|),
  so one-hot coefficients give kappa(s) / kappa(0) = phi^m(|s|) / phi^m(0) at
  |s|^2 = 1, 2, 3, and the unit-norm basis fixes kappa(0) itself.

A truncating rounding, a missing factor 1/2 or eps in place of eps^2 in the
exponent fails these tests.
"""
import numpy as np
import pytest
import torch

from oracle import basis, conv
from workloads.configs import LayerSpec


def _f32(bits):
    return np.array(bits, np.uint32).view(np.float32)


def _bits(x):
    return np.asarray(x, np.float32).view(np.uint32)


# (input float32 bit pattern, expected bfloat16 pattern in the upper half), worked out by hand:
# bfloat16 keeps the upper 16 bits; the lower 16 decide the rounding (ties to an even upper half).
RNE_CASES = [
    (0x3F800000, 0x3F80),  # 1                  exact
    (0x3F808000, 0x3F80),  # 1 + 2^-8           tie, 0x3F80 is even -> down
    (0x3F818000, 0x3F82),  # 1 + 3*2^-8         tie, 0x3F81 is odd -> up to 1 + 2^-6
    (0x3F808001, 0x3F81),  # just above the tie -> up
    (0x3F807FFF, 0x3F80),  # just below the tie -> down
    (0x3F81FFFF, 0x3F82),  # 1 + 2^-7 + (almost 2^-7) -> up
    (0xBF808000, 0xBF80),  # -(1 + 2^-8)        tie -> -1
    (0xBF818000, 0xBF82),  # -(1 + 3*2^-8)      tie -> -(1 + 2^-6)
    (0xBF808001, 0xBF81),  # negative, above the tie in magnitude -> away from zero
    (0x00000000, 0x0000),  # +0
    (0x80000000, 0x8000),  # -0
    (0x00008000, 0x0000),  # smallest subnormal tie (2^-134 + ...) -> even (0)
    (0x00018000, 0x0002),  # subnormal tie from an odd upper half -> up
    (0x7F7F7FFF, 0x7F7F),  # below the tie under the largest bfloat16 -> stays finite
    (0x7F7F8000, 0x7F80),  # tie above the largest bfloat16 (odd 0x7F7F) -> overflows to +inf
    (0x7F7FFFFF, 0x7F80),  # the largest float32 -> +inf
    (0xFF7FFFFF, 0xFF80),  # the most negative float32 -> -inf
    (0x7F800000, 0x7F80),  # +inf stays
    (0xFF800000, 0xFF80),  # -inf stays
]


@pytest.mark.parametrize("src,want", RNE_CASES)
def test_round_bf16_literal_cases(src, want):
    got = conv.round_bf16(_f32([src]))
    assert got.dtype == np.float64
    assert _bits(got)[0] == np.uint32(want << 16), (hex(src), hex(int(_bits(got)[0])), hex(want << 16))


def test_round_bf16_keeps_nan():
    got = conv.round_bf16(_f32([0x7FC00000, 0xFFC00001]))
    assert np.isnan(got).all()


def test_round_bf16_matches_torch_on_random_values():
    rng = np.random.default_rng(20211107)
    # uniformly random bit patterns (every exponent, both signs, subnormals) with NaN removed,
    # plus normal values of moderate size and values exactly on a rounding tie
    bits = rng.integers(0, 1 << 32, 1_000_000, dtype=np.uint64).astype(np.uint32)
    x = bits.view(np.float32)
    x = x[~np.isnan(x)]
    y = rng.standard_normal(200_000).astype(np.float32) * np.float32(1e3)
    ties = ((rng.integers(0, 1 << 16, 50_000, dtype=np.uint32) << 16) | np.uint32(0x8000)).view(np.float32)
    ties = ties[~np.isnan(ties)]
    for v in (x, y, ties):
        want = torch.from_numpy(v.copy()).to(torch.bfloat16).to(torch.float64).numpy()
        got = conv.round_bf16(v)
        same = (got == want) | (np.isnan(got) & np.isnan(want))
        assert same.all(), (v[~same][:5], got[~same][:5], want[~same][:5])


def test_round_bf16_is_shape_preserving_and_idempotent():
    x = np.random.default_rng(3).standard_normal((4, 5, 6))
    r = conv.round_bf16(x)
    assert r.shape == x.shape
    assert (conv.round_bf16(r) == r).all()
    # at most half a bfloat16 ulp away (relative 2^-8 for normal values)
    assert (np.abs(r - x) <= np.abs(x) * 2.0 ** -8 * (1 + 1e-12)).all()


# phi^m(r) for eps = 0.6, i.e. exp(-(r - m)^2 / 0.72), at the 3x3x3 offset radii
EXP_M0 = {1: 0.249352208777296198818257684395,     # exp(-1 / 0.72)
          2: 0.0621765240221163114948684693312,    # exp(-2 / 0.72)
          3: 0.0155038535990093188821843289062}    # exp(-3 / 0.72)
RATIO_M1 = {1: 4.01039158587574193257619584746,    # phi^1(1) / phi^1(0)
            2: 3.16006699655065129094187291883,    # phi^1(sqrt 2) / phi^1(0)
            3: 1.90519730726013649148268256083}    # phi^1(sqrt 3) / phi^1(0)
# kappa(0) of the unit-Frobenius-norm basis element on the 27 offsets:
# phi(0) / sqrt(sum_s phi(|s|)^2) for m = 0 and m = 1
KAPPA0 = {0: 0.838775907661671213446341460321, 1: 0.0637097853268695930557974332324}


def test_radial_literal_values():
    r = np.array([1.0, np.sqrt(2.0), np.sqrt(3.0)])
    np.testing.assert_allclose(basis.radial(r, 0.0, 0.6), [EXP_M0[1], EXP_M0[2], EXP_M0[3]], rtol=1e-14)
    np.testing.assert_allclose(basis.radial(r, 1.0, 0.6) / basis.radial(np.array([0.0]), 1.0, 0.6),
                               [RATIO_M1[1], RATIO_M1[2], RATIO_M1[3]], rtol=1e-14)
    assert basis.radial(np.array([2.5]), 2.5, 0.6)[0] == 1.0


@pytest.mark.parametrize("m", [0, 1])
def test_isotropic_stencil_follows_the_radial_profile(m):
    # one scalar field in and out, 3x3x3, shells {0, 1}: coefficients (J = 0, shell 0), (J = 0, shell 1)
    spec = LayerSpec(3, 1, True, ((0, 1),), ((0, 1),), shells=(0.0, 1.0))
    lay = conv.Layer(spec)
    assert lay.n_coeff == 2
    w = np.zeros(2)
    w[m] = 1.0
    kap = lay.kappa(w)[:, 0, 0]                    # [27]
    r2 = (basis.offsets(3) ** 2).sum(1)
    centre = int(np.flatnonzero(r2 == 0)[0])
    assert abs(kap[centre] - KAPPA0[m]) < 1e-14
    want = EXP_M0 if m == 0 else RATIO_M1
    for v in (1, 2, 3):
        np.testing.assert_allclose(kap[r2 == v] / kap[centre], want[v], rtol=1e-13)

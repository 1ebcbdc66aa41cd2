"""The gradient criterion of tests/parity.py on constructed cases (no GPU): a bfloat16 gradient
passes when it is the round-to-nearest-even of a value within the float32 tolerance of the
float64 gradient, and fails when it is the other neighbour away from a rounding midpoint."""

import numpy as np

from oracle import cis as O
from tests import parity as P


def _bits(x):
    return O.bf16_bits_to_float64(O.round_float64_to_bf16_bits(np.asarray(x, dtype=np.float64)))


def _next_up(x):
    """The bfloat16 neighbour of RNE(x) one step further from zero."""
    b = O.round_float64_to_bf16_bits(np.array([x], dtype=np.float64)).astype(np.int64) + 1
    return float(O.bf16_bits_to_float64(b.astype(np.uint16))[0])


def test_correctly_rounded_gradient_passes():
    rng = np.random.default_rng(0)
    g64 = rng.standard_normal((4, 257)) * 10.0 ** rng.uniform(-8, 0, (4, 257))
    st = P.grad_stats(_bits(g64), g64, bf16=True)
    assert st["out_of_tolerance"] == 0 and st["bit_equal"] == g64.size
    assert st["max_row_rel_l2"] == 0.0


def test_other_neighbour_away_from_a_midpoint_fails():
    g64 = np.array([[1.0 + 2.0 ** -10, 0.25, -3.0]])   # a quarter ulp above 1: no midpoint near
    g = _bits(g64)
    g[0, 0] = _next_up(g64[0, 0])
    st = P.grad_stats(g, g64, bf16=True)
    assert st["out_of_tolerance"] == 1


def test_other_neighbour_at_a_midpoint_passes():
    # exactly between 1 and 1 + 2^-7, nudged by 1e-6 relative: inside the float32 band
    mid = 1.0 + 2.0 ** -8
    g64 = np.array([[mid * (1 + 1e-6), mid * (1 - 1e-6), 0.5]])
    for pick in (1.0, 1.0 + 2.0 ** -7):
        g = _bits(g64)
        g[0, 0] = pick
        g[0, 1] = pick
        st = P.grad_stats(g, g64, bf16=True)
        assert st["out_of_tolerance"] == 0
        assert st["midpoint_band"] == 2
        # the row's norm sits in the two band elements: over all elements it exceeds 2e-3,
        # over the elements outside the bands it is 0
        assert st["max_row_rel_l2"] == 0.0


def test_flush_to_zero_below_float32_normals():
    g64 = np.array([[2.0 ** -127, -2.0 ** -130, 1.0]])
    g = np.array([[0.0, -0.0, 1.0]])
    assert P.grad_stats(g, g64, bf16=True)["out_of_tolerance"] == 0
    g64 = np.array([[2.0 ** -120, 1.0]])
    assert P.grad_stats(np.array([[0.0, 1.0]]), g64, bf16=True)["out_of_tolerance"] == 1


def test_float32_gradients():
    g64 = np.array([[1.0, -2.5e-3, 7.0e-20]])
    g = g64 * (1 + 1.5e-5)
    assert P.grad_stats(g, g64, bf16=False)["out_of_tolerance"] == 0
    g = g64 * (1 + 3e-5)
    assert P.grad_stats(g, g64, bf16=False)["out_of_tolerance"] == 3

"""Pins of the oracle's float64 -> bfloat16 rounding (round to nearest, ties to even).

The gradient reference rounds the float64 gradient straight to bfloat16. These checks compare
that routine with torch's float32 -> bfloat16 conversion on float32-representable inputs (where
the two must agree) and with hand-constructed ties, double-rounding, overflow and subnormal
cases whose correct results follow from the bfloat16 format itself.
"""

import math

import numpy as np
import torch

import oracle.cis as O


def torch_bf16_bits(x32: np.ndarray) -> np.ndarray:
    t = torch.from_numpy(x32.astype(np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def test_matches_torch_on_float32_inputs():
    rng = np.random.default_rng(0)
    x = np.concatenate([
        rng.normal(0, 1, 200000),
        rng.normal(0, 1, 20000) * 1e-30,
        rng.normal(0, 1, 20000) * 1e30,
        (rng.normal(0, 1, 20000) * 1e-39),          # float32 subnormals
        np.array([0.0, -0.0, 1.0, -1.0, 3.3895313892515355e38]),
    ]).astype(np.float32)
    # include exact bfloat16 midpoints (bit 15 set, lower bits clear) of both parities
    mids = (rng.integers(0x00800000, 0x7F000000, 20000, dtype=np.uint32) & np.uint32(0xFFFF0000)) \
        | np.uint32(0x8000)
    x = np.concatenate([x, mids.view(np.float32), (-mids.view(np.float32))])
    got = O.round_float64_to_bf16_bits(x.astype(np.float64))
    ref = torch_bf16_bits(x)
    assert np.array_equal(got, ref)


def test_direct_rounding_from_float64_avoids_double_rounding():
    # 1 + 2^-8 + 2^-30: above the midpoint between 1 and 1 + 2^-7, so it rounds up; a detour
    # through float32 lands exactly on the midpoint and then ties to 1.0
    x = 1.0 + 2.0 ** -8 + 2.0 ** -30
    assert O.bf16_bits_to_float64(O.round_float64_to_bf16_bits(np.array([x])))[0] == 1.0 + 2.0 ** -7
    assert float(np.float32(x)) == 1.0 + 2.0 ** -8


def test_ties_to_even_overflow_subnormals():
    cases = {
        1.0 + 2.0 ** -8: 1.0,                                # tie -> even (1.0)
        1.0 + 3 * 2.0 ** -8: 1.0 + 2.0 ** -6,                # tie -> even (upper)
        -(1.0 + 2.0 ** -8): -1.0,
        math.ldexp(2.0 - 2.0 ** -7, 127): math.ldexp(2.0 - 2.0 ** -7, 127),
        math.ldexp(2.0 - 2.0 ** -8, 127): math.inf,          # tie above max finite -> inf
        math.ldexp(2.0 - 2.0 ** -8 - 2.0 ** -20, 127): math.ldexp(2.0 - 2.0 ** -7, 127),
        0.5 * 2.0 ** -133: 0.0,                              # tie between 0 and min subnormal
        0.75 * 2.0 ** -133: 2.0 ** -133,
        1.5 * 2.0 ** -133: 2.0 * 2.0 ** -133,                # tie -> even
        2.0 ** -126 * (1 - 2.0 ** -9): 2.0 ** -126,          # rounds up into the normal range
    }
    xs = np.array(list(cases.keys()))
    got = O.bf16_bits_to_float64(O.round_float64_to_bf16_bits(xs))
    for x, g in zip(xs, got):
        assert g == cases[float(x)], (x, g, cases[float(x)])
    nanb = O.round_float64_to_bf16_bits(np.array([math.nan]))[0]
    assert (nanb & 0x7F80) == 0x7F80 and (nanb & 0x7F) != 0


def test_neighbors_bracket_and_are_adjacent():
    rng = np.random.default_rng(1)
    x = np.concatenate([rng.normal(0, 1, 5000), rng.normal(0, 1, 500) * 1e-39,
                        np.array([0.0, 1.0, -2.0, 1e-45, -1e-45])])
    lo, hi = O.bf16_neighbors(x)
    assert np.all(lo <= x) and np.all(x <= hi)
    rep = O.bf16_bits_to_float64(O.round_float64_to_bf16_bits(x)) == x
    assert np.all((lo == hi) == rep)
    # adjacent: no bfloat16 strictly between lo and hi (check via the midpoint rounding)
    mid = 0.5 * (lo + hi)
    r = O.bf16_bits_to_float64(O.round_float64_to_bf16_bits(mid))
    assert np.all((r == lo) | (r == hi))


def test_bf16_matrix_rows_match_torch_conversion():
    rng = np.random.default_rng(2)
    x = torch.from_numpy(rng.normal(0, 5, (7, 301)).astype(np.float32)).to(torch.bfloat16)
    x[0, :5] = torch.tensor([float("inf"), -float("inf"), 0.0, -0.0, 3.0e38])
    bits = x.view(torch.int16).numpy().view(np.uint16)
    m = O.Bf16Matrix(bits)
    assert m.shape == (7, 301)
    ref = x.to(torch.float64).numpy()
    for t in range(7):
        row = m[t]
        assert row.dtype == np.float64
        assert np.array_equal(row, ref[t]) and np.array_equal(np.signbit(row), np.signbit(ref[t]))

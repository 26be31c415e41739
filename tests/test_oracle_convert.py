"""Pins of the oracle's 32 <-> 16-bit converter (section 5.5) against facts
that do not come from its own code:

  - the bit layout: dropping 16 fraction bits keeps the high half of the
    fp32 pattern, checked on every one of the 2**32 inputs (NaN excepted,
    which the reading maps to the quiet NaN of its sign);
  - order facts of rounding toward zero, on random values of every
    magnitude: the result is at most |x| in magnitude, has x's sign, and the
    next 16-bit value away from zero is above |x|;
  - the relative error bound 2**-7 of an 8-significant-bit truncation;
  - special values and the subnormal quantum;
  - widening then converting is the identity on every 16-bit pattern.
"""

import concurrent.futures

import numpy as np
import pytest

from oracle import convert

SLICE = 1 << 24


def _bit_formula(u: np.ndarray) -> np.ndarray:
    hi = (u >> np.uint32(16)).astype(np.uint16)
    nan = ((u & np.uint32(0x7F800000)) == np.uint32(0x7F800000)) & ((u & np.uint32(0x007FFFFF)) != 0)
    canon = np.where((u >> np.uint32(31)) != 0, np.uint16(0xFFC0), np.uint16(0x7FC0)).astype(np.uint16)
    return np.where(nan, canon, hi)


def _check_slice(first: int) -> int:
    got = convert.truncate_bf16_range(first, SLICE)
    u = np.arange(first, first + SLICE, dtype=np.uint64).astype(np.uint32)
    bad = np.flatnonzero(got != _bit_formula(u))
    return int(bad.size) if bad.size == 0 else int(u[bad[0]])


def test_converter_matches_the_bit_layout_on_all_2_32_inputs():
    firsts = list(range(0, 1 << 32, SLICE))
    with concurrent.futures.ThreadPoolExecutor(max_workers=8) as ex:
        results = list(ex.map(_check_slice, firsts))
    bad = [(f, r) for f, r in zip(firsts, results) if r != 0]
    assert not bad, f"first mismatching input pattern: {bad[0][1]:#010x}"


def test_rounding_toward_zero_order_facts():
    rng = np.random.default_rng(0)
    # every exponent, random fractions, both signs
    u = rng.integers(0, 1 << 32, size=1 << 20, dtype=np.uint64).astype(np.uint32)
    x = u.view(np.float32)
    x = x[np.isfinite(x)]
    t = convert.truncate_bf16(x.astype(np.float64))
    xd = x.astype(np.float64)
    assert np.all(np.abs(t) <= np.abs(xd))
    assert np.all((t == 0) | (np.sign(t) == np.sign(xd)))
    # next value away from zero in the 16-bit format is above |x|
    bits = convert.truncate_bf16_bits(x)
    mag = (bits & np.uint16(0x7FFF)).astype(np.uint32)
    nxt = convert.widen_bf16(mag + 1)  # magnitude one step up (0x7F80 = inf at the top)
    assert np.all(nxt > np.abs(xd))
    # relative error below 2^-7 in the normal range
    normal = np.abs(xd) >= 2.0 ** -126
    rel = (np.abs(xd) - np.abs(t))[normal] / np.abs(xd)[normal]
    assert np.all(rel < 2.0 ** -7) and np.all(rel >= 0)


def test_special_values_and_subnormal_quantum():
    f = np.float32
    cases = [
        (0.0, 0x0000), (-0.0, 0x8000), (np.inf, 0x7F80), (-np.inf, 0xFF80),
        (1.0, 0x3F80), (-1.0, 0xBF80), (1.9999999, 0x3FFF), (255.99998, 0x437F),
        (float(np.finfo(np.float32).max), 0x7F7F),       # largest fp32 -> largest 16-bit value
        (2.0 ** -133, 0x0001), (2.0 ** -133 * 1.9, 0x0001), (2.0 ** -134, 0x0000),
        (2.0 ** -126 * (1 - 2.0 ** -23), 0x007F),        # largest fp32 subnormal
        (-(2.0 ** -149), 0x8000),
    ]
    for x, want in cases:
        got = int(convert.truncate_bf16_bits(np.array([x], f))[0])
        assert got == want, (x, hex(got), hex(want))
    nan = np.array([np.nan, -np.nan], f)
    nan_bits = np.array([0x7F800001, 0xFF800001, 0x7FC00000, 0x7FFFFFFF], np.uint32).view(np.float32)
    got = convert.truncate_bf16_bits(np.concatenate([nan, nan_bits]))
    assert list(got) == [0x7FC0, 0xFFC0, 0x7FC0, 0xFFC0, 0x7FC0, 0x7FC0]


def test_widen_then_convert_is_identity():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    wide = convert.widen_bf16(bits)
    back = convert.truncate_bf16_bits(wide.astype(np.float32))
    nan = np.isnan(wide)
    assert np.array_equal(back[~nan], bits[~nan])
    assert np.all((back[nan] & 0x7FFF) == 0x7FC0)
    # widening is exact: the value equals the pattern read as the top half of an fp32
    assert np.array_equal(wide[~nan].astype(np.float32).view(np.uint32) >> 16, bits[~nan].astype(np.uint32))


@pytest.mark.parametrize("x", [1.0 + 2.0 ** -8, 1.0 + 2.0 ** -8 + 2.0 ** -30, 3.0 - 2.0 ** -22])
def test_value_path_rounds_to_fp32_first(x):
    # a float64 value is first rounded to fp32 (the producer's 32-bit result),
    # then truncated: 1 + 2^-8 + 2^-30 rounds to 1 + 2^-8 in fp32
    t = convert.truncate_bf16(np.array([x]))[0]
    f = float(np.float32(x))
    want = np.floor(f * 128.0) / 128.0 if 1.0 <= f < 2.0 else np.floor(f * 64.0) / 64.0
    assert t == want


def test_truncating_step_stores_values_rounded_toward_zero():
    import oracle
    rng = np.random.default_rng(5)
    x = oracle.round_bf16(rng.standard_normal((9, 6)))
    masters = [rng.standard_normal((6, 7)) * 0.3, rng.standard_normal((7, 4)) * 0.3]
    masters = [m.astype(np.float32).astype(np.float64) for m in masters]
    weights = [oracle.round_to(m, "bf16t") for m in masters]
    biases = [rng.standard_normal(7) * 0.1, rng.standard_normal(4) * 0.1]
    biases = [b.astype(np.float32).astype(np.float64) for b in biases]
    target = oracle.round_bf16(rng.standard_normal((9, 4)))
    ref = oracle.dense_step(x, weights, biases, [True, False], act="bf16", target=target, masters=masters,
                            rounding="truncate")
    near = oracle.dense_step(x, weights, biases, [True, False], act="bf16", target=target, masters=masters)
    for t in ref["h"][1:] + ref["dx"] + ref["new_weights"]:
        assert np.array_equal(oracle.round_bf16(t), t)       # representable in 16 bits
    # layer 1 from the same operands: truncation toward zero of the fp32 result
    y = oracle.matmul(x, weights[0], out="f32", bias=biases[0], relu=True)
    assert np.all(np.abs(ref["h"][1]) <= y) and np.all(y - ref["h"][1] < 2.0 ** -7 * y + 1e-300)
    assert np.all(np.abs(near["h"][1] - y) <= 2.0 ** -8 * y)
    # the 16-bit weight copies are the updated masters truncated
    for m, w16 in zip(ref["new_masters"], ref["new_weights"]):
        assert np.all(np.abs(w16) <= np.abs(m)) and np.all(np.abs(m - w16) < 2.0 ** -7 * np.abs(m) + 1e-300)

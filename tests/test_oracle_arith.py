"""Pins of the oracle's arithmetic: the binary16 cast, binary16 add, and divide-by-N.

Against hand-worked cases (tests/golden/rounding.txt), an integer implementation of
round-to-nearest-even written from the IEEE-754 definition, torch's independent
CPU conversion, and binary64 arithmetic with one final rounding.
"""
import numpy as np
import torch

import _pins
from oracle import fusion, ring


def f32_to_f16_ref(bits):
    """binary32 bit patterns -> binary16 bit patterns, round to nearest even, gradual
    underflow, overflow to infinity; integer arithmetic only.  NaN inputs excluded.

    The input is M * 2^E exactly.  binary16's quantum at that magnitude is 2^Q with
    Q = floor(log2 |x|) - 10 in the normal range and 2^-24 below 2^-14.  M is rounded to
    a multiple of the quantum (ties to the even multiple) and re-encoded; the encoding
    ((Q + 25) << 10) + q - 1024 also covers the carry into the next binade and the
    subnormal range, and anything at or above 0x7c00 is infinity.
    """
    b = np.asarray(bits, dtype=np.uint32).astype(np.int64)
    sign = (b >> 31) << 15
    e = (b >> 23) & 0xFF
    m = b & 0x7FFFFF
    M = np.where(e == 0, m, m | 0x800000)
    E = np.where(e == 0, -149, e - 150)
    lead = np.where(e == 0, -200, e - 127)
    Q = np.where(lead >= -14, lead - 10, -24)
    shift = np.minimum(Q - E, 40)
    q = M >> shift
    r = M - (q << shift)
    half = np.int64(1) << (shift - 1)
    q = q + ((r > half) | ((r == half) & ((q & 1) == 1)))
    h = ((Q + 25) << 10) + q - 1024
    h = np.minimum(h, 0x7C00)
    return (sign | h).astype(np.uint16)


def _structured_f32_patterns():
    """Every combination of the top 24 bits with low bytes 0x00, 0x01, 0x80, 0xff:
    covers exact ties, one past them, and every binade and fp16 quantum."""
    top = np.arange(1 << 24, dtype=np.uint32) << np.uint32(8)
    return np.concatenate([top | np.uint32(lo) for lo in (0x00, 0x01, 0x80, 0xFF)])


def test_golden_rounding_table():
    rows = _pins.read_rounding_golden()
    assert len(rows) >= 30
    for row in rows:
        kind = row[0]
        if kind == "cast":
            got = fusion.cast(_pins.f32_bits(row[1]), np.float16)
            assert _pins.bits_equal(got, _pins.f16_bits(row[2])), row
        elif kind == "add16":
            got = ring.add(_pins.f16_bits(row[1]), _pins.f16_bits(row[2]))
            assert _pins.bits_equal(got, _pins.f16_bits(row[3])), row
        elif kind == "div32":
            got = ring.divide(_pins.f32_bits(row[1]), int(row[2]))
            assert _pins.bits_equal(got, _pins.f32_bits(row[3])), row
        elif kind == "div16":
            got = ring.divide(_pins.f16_bits(row[1]), int(row[2]))
            assert _pins.bits_equal(got, _pins.f16_bits(row[3])), row
        else:
            raise AssertionError(row)


def test_integer_reference_reproduces_golden_casts():
    for row in _pins.read_rounding_golden():
        if row[0] == "cast":
            assert int(f32_to_f16_ref(np.array([int(row[1], 16)]))[0]) == int(row[2], 16), row


def test_cast_to_fp16_structured_patterns():
    pats = _structured_f32_patterns()
    exp = (pats >> np.uint32(23)) & np.uint32(0xFF)
    man = pats & np.uint32(0x7FFFFF)
    pats = pats[~((exp == 0xFF) & (man != 0))]  # drop NaNs
    for lo in range(0, pats.size, 1 << 24):
        p = pats[lo : lo + (1 << 24)]
        got = fusion.cast(p.view(np.float32), np.float16).view(np.uint16)
        assert np.array_equal(got, f32_to_f16_ref(p))
        if lo == 0:
            tor = torch.from_numpy(p.view(np.float32)).to(torch.float16).view(torch.int16).numpy().view(np.uint16)
            assert np.array_equal(got, tor)


def test_widen_fp16_exact():
    h = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    h = h[(h & 0x7C00) != 0x7C00]  # finite values
    w = fusion.cast(h.view(np.float16), np.float32)
    back = fusion.cast(w, np.float16)
    assert np.array_equal(back.view(np.uint16), h)
    # the value: (-1)^s * 2^(e-15) * (1 + m/1024), or 2^-24 * m when e == 0
    s = (h >> 15).astype(np.int64)
    e = ((h >> 10) & 0x1F).astype(np.int64)
    m = (h & 0x3FF).astype(np.int64)
    val = np.where(e == 0, m * 2.0 ** -24, (1024 + m) * np.ldexp(1.0, (e - 25).astype(np.int32)))
    assert np.array_equal(w.astype(np.float64), np.where(s == 1, -val, val))


def test_fp16_add_equals_single_rounding_of_exact_sum():
    """Every finite binary16 a against 257 chosen b, plus 4M random pairs: the oracle's
    add equals the exact sum (exact in binary64) rounded once."""
    allh = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    allh = allh[(allh & 0x7C00) != 0x7C00].view(np.float16)
    rng = np.random.default_rng(11)
    picks = np.concatenate([allh[:: 256], _pins.f16_bits("0001"), _pins.f16_bits("8001"), _pins.f16_bits("3c00")])
    for b in picks:
        bb = np.full(allh.shape, b, dtype=np.float16)
        got = ring.add(allh, bb)
        want = _pins.add_ref(allh, bb)
        ok = np.isnan(want) | (got.view(np.uint16) == want.view(np.uint16))
        assert np.all(ok)
    a = rng.choice(allh, 1 << 22)
    b = rng.choice(allh, 1 << 22)
    got, want = ring.add(a, b), _pins.add_ref(a, b)
    assert np.array_equal(got.view(np.uint16), want.view(np.uint16))


def test_divide_equals_single_rounding_of_exact_quotient():
    rng = np.random.default_rng(12)
    x32 = (rng.standard_normal(1 << 20) * rng.choice([1e-30, 1e-3, 1.0, 1e20], 1 << 20)).astype(np.float32)
    allh = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    x16 = allh[(allh & 0x7C00) != 0x7C00].view(np.float16)
    for n in list(range(1, 70)) + [128, 1000]:
        assert _pins.bits_equal(ring.divide(x32, n), _pins.div_ref(x32, n)), n
        assert _pins.bits_equal(ring.divide(x16, n), _pins.div_ref(x16, n)), n


def test_fp32_add_equals_single_rounding():
    rng = np.random.default_rng(13)
    a = (rng.standard_normal(1 << 20) * rng.choice([1e-8, 1e-2, 1.0, 1e6], 1 << 20)).astype(np.float32)
    b = (rng.standard_normal(1 << 20) * rng.choice([1e-8, 1e-2, 1.0, 1e6], 1 << 20)).astype(np.float32)
    assert _pins.bits_equal(ring.add(a, b), _pins.add_ref(a, b))

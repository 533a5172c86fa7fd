"""The oracle's bf16 decoding, pinned by values fixed outside the oracle.

bf16 is the upper half of an IEEE-754 binary32: 1 sign bit, 8 exponent bits
(bias 127) and 7 stored fraction bits. The attention inputs (Q, K, V) and the
ragged workload's logits arrive as raw bf16 bit patterns, and both
`oracle.attention.decode_bf16` and the bf16 branch of
`oracle.accept.decode_logits` turn them into fp64 values. The checks here do
not go through binary32 at all: hand-written patterns with their known values,
and every one of the 65536 patterns against the field formula
(-1)^s * 2^(e - 127) * (1 + f / 128) (normal), (-1)^s * 2^-126 * (f / 128)
(subnormal), +-inf and NaN, evaluated with exact integer/`ldexp` arithmetic.
"""

import math

import numpy as np
import pytest

from oracle.accept import decode_logits
from oracle.attention import decode_bf16

# (bit pattern, exact value)
HAND = [
    (0x3F80, 1.0),
    (0xC000, -2.0),
    (0x0000, 0.0),
    (0x8000, -0.0),
    (0x0001, 2.0 ** -133),           # smallest subnormal: 2^-126 * 2^-7
    (0x007F, 127 * 2.0 ** -133),     # largest subnormal
    (0x0080, 2.0 ** -126),           # smallest normal
    (0x7F80, math.inf),
    (0xFF80, -math.inf),
    (0x4049, 3.140625),              # 2 * (1 + 73/128)
    (0x3F81, 1.0 + 2.0 ** -7),
    (0xBF40, -0.75),
    (0x7F7F, (2.0 - 2.0 ** -7) * 2.0 ** 127),  # largest finite
    (0x4110, 9.0),
    (0xC2F7, -123.5),
]

DECODERS = [("decode_bf16", decode_bf16), ("decode_logits", decode_logits)]


def field_value(bits: int) -> float:
    """The value a bf16 pattern encodes, from its three fields."""
    s = -1.0 if bits & 0x8000 else 1.0
    e = (bits >> 7) & 0xFF
    f = bits & 0x7F
    if e == 0xFF:
        return s * math.inf if f == 0 else math.nan
    if e == 0:
        return s * math.ldexp(f, -126 - 7)
    return s * math.ldexp(128 + f, e - 127 - 7)


@pytest.mark.parametrize("name,fn", DECODERS, ids=[d[0] for d in DECODERS])
def test_hand_written_patterns(name, fn):
    bits = np.array([b for b, _ in HAND], dtype=np.uint16)
    got = fn(bits)
    assert got.dtype == np.float64
    for (b, want), g in zip(HAND, got):
        assert g == want, f"{name}(0x{b:04X}) = {g!r}, want {want!r}"
        assert math.copysign(1.0, g) == math.copysign(1.0, want), f"{name}(0x{b:04X}) sign"


@pytest.mark.parametrize("name,fn", DECODERS, ids=[d[0] for d in DECODERS])
def test_every_pattern_against_field_formula(name, fn):
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    with np.errstate(invalid="ignore"):  # signalling-NaN patterns widen to quiet NaNs
        got = fn(bits)
    want = np.array([field_value(int(b)) for b in range(1 << 16)], dtype=np.float64)
    nan_w = np.isnan(want)
    assert (np.isnan(got) == nan_w).all()
    np.testing.assert_array_equal(got[~nan_w], want[~nan_w])
    assert (np.signbit(got[~nan_w]) == np.signbit(want[~nan_w])).all()


@pytest.mark.parametrize("name,fn", DECODERS, ids=[d[0] for d in DECODERS])
def test_shape_and_multidimensional_input(name, fn):
    bits = np.array([[0x3F80, 0xC000], [0x4049, 0xBF40]], dtype=np.uint16)
    got = fn(bits)
    assert got.shape == (2, 2)
    np.testing.assert_array_equal(got, [[1.0, -2.0], [3.140625, -0.75]])


def test_fp32_logits_pass_through_exactly():
    x = np.array([1.5, -3.25e-20, np.float32(1e30), -np.inf], dtype=np.float32)
    got = decode_logits(x)
    assert got.dtype == np.float64
    np.testing.assert_array_equal(got, x.astype(np.float64))

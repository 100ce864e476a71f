"""Pins for the oracle's fp16 / bf16 storage conversions.

The oracle's encoders are written from the IEEE 754 definitions; here they
are checked against independent library conversions (numpy's float64 ->
float16 and torch's float32 -> bfloat16, both round-to-nearest-even) and
against hand-derived boundary values.
"""
import numpy as np
import pytest
import torch

import oracle


def _wide_doubles(n, seed):
    rng = np.random.default_rng(seed)
    mant = rng.uniform(-2.0, 2.0, n)
    exps = rng.integers(-30, 18, n)
    return np.ldexp(mant, exps)


def test_fp16_encode_matches_numpy():
    x = _wide_doubles(200_000, 1)
    ref = x.astype(np.float16).view(np.uint16)
    got = oracle.encode(x, "fp16")
    np.testing.assert_array_equal(got, ref)


def test_fp16_encode_boundaries():
    one = 1.0
    cases = {
        one: 0x3C00,
        one + 2.0 ** -11: 0x3C00,          # tie -> even (down)
        one + 3 * 2.0 ** -11: 0x3C02,      # tie -> even (up)
        one + 2.0 ** -11 + 2.0 ** -30: 0x3C01,   # just above the tie
        65504.0: 0x7BFF,                   # largest finite
        65519.99: 0x7BFF,
        65520.0: 0x7C00,                   # tie between 65504 and 2^16 -> overflow
        2.0 ** -24: 0x0001,                # smallest subnormal
        2.0 ** -25: 0x0000,                # tie -> even (zero)
        3 * 2.0 ** -25: 0x0002,            # tie -> even (2)
        2.0 ** -14 - 2.0 ** -25: 0x0400,   # rounds up into the normal range
        -0.0: 0x8000,
        -2.5: 0xC100,
    }
    for x, bits in cases.items():
        assert int(oracle.encode(np.array([x]), "fp16")[0]) == bits, (x, hex(bits))


def test_fp16_decode_matches_numpy():
    allbits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    finite = (allbits & 0x7C00) != 0x7C00
    ref = allbits.view(np.float16).astype(np.float64)
    got = oracle.decode(allbits, "fp16")
    np.testing.assert_array_equal(got[finite], ref[finite])
    assert np.all(np.isinf(got[(allbits & 0x7FFF) == 0x7C00]))


def test_bf16_encode_matches_torch_on_float32_values():
    # float32 inputs: torch rounds float32 -> bfloat16 to nearest even; the
    # oracle starts from the same (exactly representable) value in fp64.
    rng = np.random.default_rng(2)
    x32 = np.ldexp(rng.uniform(-2, 2, 200_000), rng.integers(-130, 120, 200_000)).astype(np.float32)
    x32 = x32[np.isfinite(x32)]
    ref = torch.from_numpy(x32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = oracle.encode(x32.astype(np.float64), "bf16")
    np.testing.assert_array_equal(got, ref)


def test_bf16_decode_is_top_half_of_float32():
    allbits = np.arange(65536, dtype=np.uint32)
    f32 = (allbits << np.uint32(16)).view(np.float32).astype(np.float64)
    got = oracle.decode(allbits.astype(np.uint16), "bf16")
    finite = np.isfinite(f32)
    np.testing.assert_array_equal(got[finite], f32[finite])


def test_bf16_boundaries():
    cases = {
        1.0 + 2.0 ** -8: 0x3F80,           # tie -> even (down)
        1.0 + 3 * 2.0 ** -8: 0x3F82,       # tie -> even (up)
        (2 - 2.0 ** -8) * 2.0 ** 127: 0x7F80,   # overflow tie -> infinity
        (2 - 2.0 ** -7) * 2.0 ** 127: 0x7F7F,   # largest finite
        2.0 ** -133: 0x0001,
    }
    for x, bits in cases.items():
        assert int(oracle.encode(np.array([x]), "bf16")[0]) == bits, (x, hex(bits))


@pytest.mark.parametrize("dtype", ["fp16", "bf16"])
def test_roundtrip_all_finite_bits(dtype):
    allbits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    v = oracle.decode(allbits, dtype)
    finite = np.isfinite(v)
    back = oracle.encode(v[finite], dtype)
    np.testing.assert_array_equal(back, allbits[finite])

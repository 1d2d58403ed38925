"""Number-format facts the int4 GEMV relies on, checked on the host (CPU).

The int4 dot product masks each stored code + 8 into the low nibble of a byte
and converts byte pairs with the FP8 E4M3 conversion: a byte n in 0..15 has
exponent field 0 or 1 (bias 7), so it reads as n * 2^-9 exactly, linear in n,
and the exact factor 2^-9 is taken out once per granule.  The high nibble in
place (byte n * 16) has no such reading, which is why the kernel shifts it
down first.  The device conversion itself is covered by the GPU parity tests.
"""
import numpy as np
import torch


def test_low_nibble_bytes_read_as_e4m3_are_exact_multiples_of_2_pow_minus_9():
    b = torch.arange(16, dtype=torch.uint8)
    v = b.view(torch.float8_e4m3fn).to(torch.float64).numpy()
    assert np.array_equal(v, np.arange(16) * 2.0 ** -9)


def test_high_nibble_bytes_in_place_are_not_linear():
    b = (torch.arange(16, dtype=torch.int32) << 4).to(torch.uint8)
    v = b.view(torch.float8_e4m3fn).to(torch.float64).numpy()
    assert not np.allclose(v, np.arange(16) * v[1])


def test_scaled_products_sum_bit_for_bit():
    """Sums of fp32 products carrying an exact factor 2^-9 equal 2^-9 times the
    plain sums bit for bit (no underflow at activation magnitudes), the property
    that keeps the FP8 reading exact against the plain conversion."""
    rng = np.random.default_rng(0)
    x = rng.standard_normal(4096).astype(np.float32)
    n = rng.integers(0, 16, 4096).astype(np.float32)
    plain = np.float32(0)
    scaled = np.float32(0)
    for a, c in zip(n, x):
        plain = np.float32(plain + np.float32(a * c))
        scaled = np.float32(scaled + np.float32(np.float32(a * np.float32(2.0 ** -9)) * c))
    assert np.float32(scaled * np.float32(512.0)) == plain

"""Host-side checks of the seeded input generator (no GPU)."""
import hashlib

import numpy as np
import pytest

from paper_2606_26344_amd import inputs as I


def _bits(x):
    return [int(v) for v in I.f32_to_bf16_bits(np.array(x, dtype=np.float32))]


def test_bf16_round_to_nearest_even():
    # 1 + 2^-8 is exactly half an ulp above 1.0: ties go to the even mantissa.
    assert _bits([1.0 + 2.0 ** -8]) == [0x3F80]
    # 1 + 3 * 2^-8 is half an ulp above 0x3F81 (odd): rounds up to 0x3F82.
    assert _bits([1.0 + 3 * 2.0 ** -8]) == [0x3F82]
    assert _bits([1.0 + 0.75 * 2.0 ** -7]) == [0x3F81]
    assert _bits([1.0 + 0.375 * 2.0 ** -7]) == [0x3F80]
    assert _bits([-2.5]) == [0xC020]


def test_bf16_special_values():
    assert _bits([0.0, -0.0]) == [0x0000, 0x8000]
    assert _bits([np.inf, -np.inf]) == [0x7F80, 0xFF80]
    nan = _bits([np.nan])[0]
    assert (nan & 0x7F80) == 0x7F80 and (nan & 0x007F) != 0
    # Largest finite float32 rounds past the bf16 range to +inf.
    assert _bits([np.finfo(np.float32).max]) == [0x7F80]
    # Subnormals are kept (no flush to zero).
    assert _bits([1e-40]) == [0x0001]
    assert _bits([np.float32(2.0 ** -133)]) == [0x0001]  # smallest bf16 subnormal
    assert _bits([np.float32(2.0 ** -135)]) == [0x0000]  # a quarter of it


def test_bf16_decode_is_exact_inverse_on_bf16_values():
    bits = np.arange(0, 1 << 16, dtype=np.uint32).astype(np.uint16)
    vals = I.bf16_bits_to_f32(bits)
    finite = np.isfinite(vals)
    again = I.f32_to_bf16_bits(vals[finite])
    assert np.array_equal(again, bits[finite])


def test_generator_is_deterministic_and_seeded():
    a = I.generate(16, 256, 512, seed=0)
    b = I.generate(16, 256, 512, seed=0)
    c = I.generate(16, 256, 512, seed=1)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
    assert not np.array_equal(a[1], c[1])


def test_generator_shapes_and_scales():
    X, Wg, Wu, Wd = I.generate(8, 512, 1024, seed=0)
    assert X.shape == (8, 512) and Wg.shape == (512, 1024)
    assert Wu.shape == (512, 1024) and Wd.shape == (1024, 512)
    assert all(m.dtype == np.uint16 for m in (X, Wg, Wu, Wd))
    # variance 1 / fan_in
    assert abs(I.bf16_bits_to_f32(Wg).std() * np.sqrt(512) - 1.0) < 0.02
    assert abs(I.bf16_bits_to_f32(Wd).std() * np.sqrt(1024) - 1.0) < 0.02
    assert abs(I.bf16_bits_to_f32(X).std() - 1.0) < 0.05


def test_unit_rms_rows():
    X, *_ = I.generate(32, 4096, 64, seed=0, unit_rms_rows=True)
    rms = np.sqrt(np.mean(I.bf16_bits_to_f32(X).astype(np.float64) ** 2, axis=1))
    # bf16 rounding of each element moves the RMS by far less than 1e-3.
    assert np.all(np.abs(rms - 1.0) < 1e-3)


def test_tiny_workload_bytes_are_stable():
    X, Wg, Wu, Wd = I.generate_workload("tiny")
    h = hashlib.sha256()
    for m in (X, Wg, Wu, Wd):
        h.update(m.tobytes())
    # Written by this generator with numpy 2.2 (PCG64 + ziggurat float32).
    assert h.hexdigest()[:16] == TINY_SHA256_PREFIX


TINY_SHA256_PREFIX = "58ac37a2d6771f0a"


@pytest.mark.parametrize("T", [1, 100, 255, 256, 257, 4096])
def test_sample_rows(T):
    rows = I.sample_rows(T, 256)
    assert len(rows) == min(T, 256)
    assert rows.min() >= 0 and rows.max() < T
    assert np.all(np.diff(rows) > 0)
    if T > 256:
        assert {0, 1, T // 2, T - 1} <= set(rows.tolist())
        assert len({r % 32 for r in rows.tolist()}) == 32

"""The shared seeded-input module: determinism and bf16 rounding (CPU only)."""
import numpy as np

from oracle.pipeline import sampler_step
from synth import bf16_bits, bf16_round, bf16_value, normal, normal_parallel


def test_bf16_known_patterns():
    x = np.array([1.0, -2.0, 1.0 / 3.0, 0.0, 65504.0, 1e-30], dtype=np.float32)
    assert list(bf16_bits(x)) == [0x3F80, 0xC000, 0x3EAB, 0x0000, 0x4780, 0x0DA2]
    # ties go to even: 1 + 2^-8 lies halfway between 1 and 1 + 2^-7
    t = np.array([1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8], dtype=np.float32)
    assert list(bf16_bits(t)) == [0x3F80, 0x3F82]
    y = normal((1000,), (1, 2, 3))
    r = bf16_round(y)
    assert np.all(np.abs(r - y) <= np.abs(y) * 2.0 ** -8)
    np.testing.assert_array_equal(bf16_value(bf16_bits(r)), r)


def test_keys_are_order_free():
    a = normal((4, 5), (0, 1, 2))
    normal((100,), (9,))
    b = normal((4, 5), (0, 1, 2))
    np.testing.assert_array_equal(a, b)
    assert not np.array_equal(a, normal((4, 5), (0, 1, 3)))
    p1 = normal_parallel((64, 8), (4, 4), 0.02, parts=8)
    p2 = normal_parallel((64, 8), (4, 4), 0.02, parts=8)
    np.testing.assert_array_equal(p1, p2)
    assert abs(p1.std() - 0.02) < 0.005


def test_sampler_last_step_returns_prediction():
    y = normal((6, 4), (1,)).astype(np.float64)
    xi = normal((6, 4), (2,)).astype(np.float64)
    np.testing.assert_array_equal(sampler_step(y, xi, 0.0), y)
    np.testing.assert_array_equal(sampler_step(y, xi, 1.0), xi)

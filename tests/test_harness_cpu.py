"""Host pieces of the test harness that the GPU tests rely on."""
import numpy as np

import harness


def test_bfloat16_rounding_is_nearest_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -8 + 2 ** -20, -1.0 - 2 ** -8,
                  3.0e-39, 2.0 ** -126 * 1.5], np.float32)
    want = np.array([1.0, 1.0, 1.0 + 2 ** -6, 1.0 + 2 ** -7, -1.0, 3.0e-39, 2.0 ** -126 * 1.5],
                    np.float32)
    got = harness.round_to(x, "bf16")
    # every result is a bfloat16 value (low 16 bits zero)
    assert not (got.view(np.uint32) & 0xFFFF).any()
    np.testing.assert_array_equal(got[:5], want[:5])
    # the subnormal and the normal with 1 extra bit round to their neighbours
    assert abs(float(got[5]) - 3.0e-39) <= 2.0 ** -133
    assert got[6] == np.float32(2.0 ** -126 * 1.5)


def test_float16_rounding_matches_numpy():
    r = np.random.default_rng(0)
    x = (r.standard_normal(10000) * 1e-4).astype(np.float32)
    np.testing.assert_array_equal(harness.round_to(x, "f16"),
                                  x.astype(np.float16).astype(np.float32))
    assert harness.round_to(x, "f32") is not None

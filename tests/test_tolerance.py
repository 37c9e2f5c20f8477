"""The tolerance check the GPU parity tests use (tests/gpu_util.py)."""
import numpy as np
import pytest

from gpu_util import assert_close


def test_bounds_and_nan():
    ref = np.array([1.0, -2.0, 0.0, 100.0])
    assert_close(ref + np.array([1e-5, -1e-5, 1e-5, 1e-2]), ref, "f32")     # atol 1e-5 + rtol 1e-4
    with pytest.raises(AssertionError):
        assert_close(ref + np.array([0, 0, 2e-5, 0]), ref, "f32")
    for bad in (np.nan, np.inf):
        with pytest.raises(AssertionError, match="1 of 4"):
            assert_close(np.array([1.0, -2.0, bad, 100.0]), ref, "f32")
    assert_close(ref * (1 + 1.9e-2) + 9e-3, ref, "bf16")                     # atol 1e-2 + rtol 2e-2
    with pytest.raises(AssertionError):
        assert_close(np.array([1.0, -2.0, 0.0, 103.0]), ref, "bf16")

"""The element-wise parity check used by every GPU test, on the CPU: it must
reject NaN and infinite outputs (the operand padding of datagen.store is NaN,
so a kernel that reads past an operand shows up as NaN in its output) and
values outside the bound, and accept values inside it."""
import numpy as np
import pytest

import gpu_util as U


def test_accepts_within_bound():
    ref = np.array([[0.0, 1.0, -100.0]])
    got = ref + np.array([[0.0099, -0.0199, 1.0099]])
    U.assert_close(got, ref, what="inside")


@pytest.mark.parametrize("bad", [np.nan, np.inf, -np.inf])
def test_rejects_non_finite_output(bad):
    ref = np.array([[1.0, 2.0]])
    got = np.array([[1.0, bad]], dtype=np.float16)
    with pytest.raises(AssertionError):
        U.assert_close(got, ref, what="non-finite")


def test_rejects_outside_bound_and_shape_mismatch():
    ref = np.array([[1.0, 2.0]])
    with pytest.raises(AssertionError):
        U.assert_close(np.array([[1.0, 2.05]], dtype=np.float16), ref, what="outside")
    with pytest.raises(AssertionError):
        U.assert_close(np.array([1.0, 2.0], dtype=np.float16), ref, what="shape")


def test_fp16_accumulation_bound_is_looser():
    ref = np.array([[10.0]])
    got = np.array([[10.5]], dtype=np.float16)     # 0.5 <= 5e-2 + 5e-2 * 10 = 0.55
    U.assert_close(got, ref, accum="f16", what="f16")
    with pytest.raises(AssertionError):
        U.assert_close(got, ref, accum="f32", what="f32")

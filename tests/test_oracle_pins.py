"""The oracle checked against its pins (CPU only)."""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2006_12645_amd import datagen as D
import oracle_pins as P


@pytest.fixture(scope="module")
def lib():
    return O._load()


@pytest.mark.parametrize("pin", P.PINS, ids=[p.__name__ for p in P.PINS])
def test_pin(lib, pin):
    pin(lib)


def test_rejects_bad_arguments(lib):
    a = np.zeros((4, 4), np.float16)
    with pytest.raises(ValueError):
        O.gemm_bias_act(a, 2, a, 0, 4, 4, 4, lib=lib)          # bad layout
    with pytest.raises(ValueError):
        O.gemm_bias_act(a, 0, a, 0, 4, 4, 4, act=5, lib=lib)   # bad activation
    with pytest.raises(ValueError):
        O.gemm_bias_act(a, 0, a, 0, 4, 4, 4, lda=3, lib=lib)   # ld below extent
    with pytest.raises(ValueError):
        O.gemm_bias_act(a, 0, a, 0, 4, 4, 4, rows=[4], lib=lib)  # row out of range


def test_thread_count_does_not_change_result(lib):
    A, B, bias = D.random_problem(30, 37, 41, 300)
    a_st, b_st = D.store(A, D.ROW), D.store(B, D.COL)
    r1 = O.gemm_bias_act(a_st, D.ROW, b_st, D.COL, 37, 41, 300, bias=bias, nthreads=1, lib=lib)
    r8 = O.gemm_bias_act(a_st, D.ROW, b_st, D.COL, 37, 41, 300, bias=bias, nthreads=8, lib=lib)
    assert np.array_equal(r1, r8)

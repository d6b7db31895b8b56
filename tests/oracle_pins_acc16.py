"""Pins for the oracle's binary16 rounding and its fp16-accumulation
reading (the running sum rounded to binary16 after every aligned group of
32 reduction indices of each product).

Like oracle_pins.py: each ``pin_*`` takes an opened oracle library and
raises AssertionError when the library disagrees with a fact fixed by the
IEEE 754 format, by exact rational arithmetic or by a closed form.
"""
import json
import os
from fractions import Fraction

import numpy as np

from oracle import oracle as O
from paper_2006_12645_amd import datagen as D

KC = 32
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def f16(x):
    """numpy's binary64 -> binary16 conversion (round to nearest even)."""
    with np.errstate(over="ignore"):
        return float(np.float64(x).astype(np.float16))


def pin_round_f16_vs_numpy(lib):
    """Random magnitudes from subnormal to overflow, exact ties and the
    overflow threshold, against numpy's conversion."""
    rng = np.random.default_rng(41)
    xs = list(rng.standard_normal(2000) * np.exp2(rng.integers(-26, 17, size=2000)))
    # ties between neighbouring binary16 values, at several binades and in
    # the subnormal range
    for e in (-24, -20, -14, -13, -1, 0, 3, 10, 14):
        q = 2.0 ** (e - 10) if e >= -14 else 2.0 ** -24
        base = 2.0 ** e if e >= -14 else 0.0
        for m in (1, 2, 3, 5, 1023):
            xs += [base + (m + 0.5) * q, -(base + (m + 0.5) * q)]
    xs += [65504.0, 65519.99, 65520.0, -65520.0, 2.0 ** -25, 2.0 ** -25 * 1.0000001, 2.0 ** -26]
    for x in xs:
        got, want = O.round_f16(x, lib=lib), f16(x)
        assert got == want or (np.isinf(got) and np.isinf(want) and np.sign(got) == np.sign(want)), (x, got, want)


def _run(lib, A, B, la, lb, **kw):
    M, K = A.shape
    N = B.shape[1]
    return O.fused(D.store(A, la), la, D.store(B, lb), lb, M, N, K, nthreads=2, lib=lib, **kw)


def pin_acc16_single_group(lib):
    """K <= 32 is one group: the result is the exact sum rounded once to
    binary16, then the bias added exactly."""
    M, N, K = 5, 7, 29
    A, B, bias = D.random_problem(42, M, N, K)
    want = np.array([[f16(float(sum(Fraction(float(A[i, k])) * Fraction(float(B[k, j])) for k in range(K))))
                      + float(bias[j]) for j in range(N)] for i in range(M)])
    for la in (D.ROW, D.COL):
        for lb in (D.ROW, D.COL):
            got = _run(lib, A, B, la, lb, bias=bias, act=O.ACT_NONE, acc16=True)
            assert np.array_equal(got, want), (la, lb)


def pin_acc16_group_rounding_closed_form(lib):
    """A(0,k) = 64 for the first group (k < 32), a single 1 in the second
    (k = 32) and 64 again in the third (k >= 64), B = 1: the groups end at
    2048, then 2049 rounded back to 2048 (a tie, to even), then 4096, so the
    result is 4096 where the exact sum is 4097.  A variant whose second
    group adds 1 to 2047 stays exact."""
    K = 96
    a = np.zeros((1, K), np.float16)
    a[0, :32] = 64.0
    a[0, 32] = 1.0
    a[0, 64:] = 64.0
    b = np.ones((K, 1), np.float16)
    # exact: 32*64 + 1 + 32*64 = 4097.  fp16 accumulation: 2048 after the
    # first group, fp16(2049) = 2048 after the second, fp16(2048 + 2048) =
    # 4096 after the third.
    got = _run(lib, a, b, D.ROW, D.COL, act=O.ACT_NONE, acc16=True)
    assert got[0, 0] == 4096.0, got
    exact = _run(lib, a, b, D.ROW, D.COL, act=O.ACT_NONE)
    assert exact[0, 0] == 4097.0
    # variant: the first group ends at 2047 and the second adds 1 (at k = 33)
    a2 = a.copy()
    a2[0, 31] = 63.0
    a2[0, 32] = 0.0
    a2[0, 33] = 1.0
    # first group 31*64 + 63 = 2047 (exact), second 2047 + 1 = 2048, third 4096
    got = _run(lib, a2, b, D.ROW, D.COL, act=O.ACT_NONE, acc16=True)
    assert got[0, 0] == 4096.0, got


def pin_acc16_brute_force(lib):
    """Small shapes across group boundaries (K up to 80), prologue and
    second product (add and subtract), against exact rational sums rounded
    with numpy's binary16 conversion at every group end."""
    rng = np.random.default_rng(43)
    for trial in range(10):
        M, N = (int(x) for x in rng.integers(1, 5, size=2))
        K, K2 = (int(x) for x in rng.integers(1, 81, size=2))
        A, B, bias = D.random_problem(600 + trial, M, N, K, dist="uniform")
        P, Q, _ = D.random_problem(700 + trial, M, N, K2, dist="uniform")
        second = (0, 1, -1)[trial % 3]
        pro = bool(trial & 1)

        def left(x):
            v = Fraction(float(x))
            return max(v, Fraction(0)) if pro else v
        want = np.zeros((M, N))
        for i in range(M):
            for j in range(N):
                s = Fraction(0)
                for X, Y, KK, sg in ((A, B, K, 1), (P, Q, K2, second)):
                    if sg == 0:
                        continue
                    for k in range(KK):
                        s += sg * left(X[i, k]) * Fraction(float(Y[k, j]))
                        if k % KC == KC - 1 or k == KK - 1:
                            s = Fraction(f16(float(s)))
                want[i, j] = float(s) + float(bias[j])
        got = O.fused(D.store(A, D.ROW), D.ROW, D.store(B, D.COL), D.COL, M, N, K,
                      prologue_relu=pro, second=second, p_store=D.store(P, D.ROW),
                      q_store=D.store(Q, D.COL), K2=K2, bias=bias, act=O.ACT_NONE, acc16=True,
                      nthreads=2, lib=lib)
        assert np.array_equal(got, want), (trial, np.abs(got - want).max())


def pin_acc16_integer_data_is_exact(lib):
    """Integer data with every partial sum below 2048 in magnitude: every
    rounding is exact, so fp16 accumulation equals the exact sums."""
    M, N, K = 7, 9, 300
    A, B, bias = D.random_problem(44, M, N, K, dist="int")
    exact = _run(lib, A, B, D.ROW, D.COL, bias=bias, act=O.ACT_NONE)
    got = _run(lib, A, B, D.ROW, D.COL, bias=bias, act=O.ACT_NONE, acc16=True)
    assert np.array_equal(got, exact)


def golden_row(spec, K):
    """A 1 x K fp16 row from a golden case's sparse spec: keys are an index
    "k" or a range "lo:hi", values the fp16 value stored there."""
    row = np.zeros((1, K), np.float16)
    for key, v in spec.items():
        lo, _, hi = key.partition(":")
        row[0, int(lo):int(hi) if hi else int(lo) + 1] = v
    return row


def golden_acc16_sum_of_products():
    with open(os.path.join(GOLDEN, "acc16_sum_of_products.json")) as f:
        return json.load(f)["cases"]


def pin_acc16_sum_of_products_golden(lib):
    """Hand-derived binary16 results of the single running sum through A.B
    and then P.Q (tests/golden/acc16_sum_of_products.json): cancellation
    into a lower binade, a rounding inside P.Q's group, and groups aligned
    per product.  Each case is chosen so that two separate accumulators
    (Listing 5's C and R) give a different value; the binary64 path must
    give the exact one."""
    for case in golden_acc16_sum_of_products():
        K, K2 = case["K"], case["K2"]
        a, p = golden_row(case["A"], K), golden_row(case["P"], K2)
        b, q = np.ones((K, 1), np.float16), np.ones((K2, 1), np.float16)
        for la in (D.ROW, D.COL):
            for lb in (D.ROW, D.COL):
                kw = dict(second=case["second"], p_store=D.store(p, la), q_store=D.store(q, lb), K2=K2,
                          act=O.ACT_NONE, nthreads=1, lib=lib)
                got = O.fused(D.store(a, la), la, D.store(b, lb), lb, 1, 1, K, acc16=True, **kw)
                assert got[0, 0] == case["one_sum"], (case["name"], la, lb, got[0, 0])
                assert case["one_sum"] != case["two_sums"]
                ex = O.fused(D.store(a, la), la, D.store(b, lb), lb, 1, 1, K, **kw)
                assert ex[0, 0] == case["exact"], (case["name"], la, lb, ex[0, 0])


PINS = [pin_round_f16_vs_numpy, pin_acc16_single_group, pin_acc16_group_rounding_closed_form,
        pin_acc16_brute_force, pin_acc16_integer_data_is_exact, pin_acc16_sum_of_products_golden]

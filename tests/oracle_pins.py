"""Pins for the CPU oracle: checks against facts fixed by the paper's
definition and by mathematics, not against the oracle itself.

Each ``pin_*`` takes an opened oracle library (so the same battery runs on
the real oracle and on deliberately broken copies of it) and raises
AssertionError when the library disagrees with the fact it pins.

The definition pinned is the Problem Statement section's matmul followed by
the ReLU-of-add statement (Listing 1 and its expression tree), with a
length-N bias and BLAS leading dimensions.
"""
import json
import os
from fractions import Fraction

import numpy as np

from oracle import oracle as O
from paper_2006_12645_amd import datagen as D

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
LAYOUTS = [(D.ROW, D.ROW), (D.ROW, D.COL), (D.COL, D.ROW), (D.COL, D.COL)]


def run(lib, A, B, bias, la, lb, act=O.ACT_RELU, pad=0, rows=None):
    """Store logical A, B in the given layouts (optionally with padded ld)
    and evaluate the oracle."""
    M, K = A.shape
    N = B.shape[1]
    a_ext = K if la == D.ROW else M
    b_ext = N if lb == D.ROW else K
    a_st = D.store(A, la, a_ext + pad)
    b_st = D.store(B, lb, b_ext + pad)
    return O.gemm_bias_act(a_st, la, b_st, lb, M, N, K, bias=bias, act=act, rows=rows,
                           nthreads=3, lib=lib)


def pin_decoder_all_patterns(lib):
    """fp16 decoder vs numpy's binary16 -> binary64 widening on all 65536
    patterns (NaNs excluded: only their NaN-ness is checked)."""
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ref = bits.view(np.float16).astype(np.float64)
    got = np.array([O.f16_to_f64(int(b), lib=lib) for b in bits])
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])
    # sign of zero is preserved
    assert np.signbit(got[0x8000]) and not np.signbit(got[0])


def pin_golden_worked_example(lib):
    """Hand-derived 2x3x4 instance with exact values (tests/golden)."""
    g = json.load(open(os.path.join(GOLDEN, "listing1_worked_example.json")))
    A = np.array(g["A"], dtype=np.float16)
    B = np.array(g["B"], dtype=np.float16)
    bias = np.array(g["bias"], dtype=np.float16)
    for la, lb in LAYOUTS:
        pre = run(lib, A, B, bias, la, lb, act=O.ACT_NONE)
        out = run(lib, A, B, bias, la, lb, act=O.ACT_RELU)
        assert np.array_equal(pre, np.array(g["pre_activation"])), (la, lb, pre)
        assert np.array_equal(out, np.array(g["relu_output"])), (la, lb, out)


def pin_all_ones(lib):
    """A = B = 1: every pre-activation is K + bias[j] (exact)."""
    M, N, K = 5, 7, 33
    A = np.ones((M, K), np.float16)
    B = np.ones((K, N), np.float16)
    bias = D.uniform_f16(11, (N,))
    want = np.broadcast_to(K + bias.astype(np.float64), (M, N))
    for la, lb in LAYOUTS:
        assert np.array_equal(run(lib, A, B, bias, la, lb), want), (la, lb)


def pin_identity(lib):
    """A = I (M = K): out(i,j) = relu(B(i,j) + bias[j]); the fp64 sum of two
    fp16 values is exact."""
    n, N = 16, 9
    A = np.eye(n, dtype=np.float16)
    B = D.uniform_f16(12, (n, N), -4, 4)
    bias = D.uniform_f16(13, (N,))
    want = np.maximum(B.astype(np.float64) + bias.astype(np.float64), 0.0)
    for la, lb in LAYOUTS:
        assert np.array_equal(run(lib, A, B, bias, la, lb), want), (la, lb)


def pin_rank1(lib):
    """K = 1: out = relu(u_i * v_j + bias_j); the fp16 product is exact in
    binary64, so only the bias add rounds."""
    M, N = 6, 10
    u = D.uniform_f16(14, (M, 1), -8, 8)
    v = D.uniform_f16(15, (1, N), -8, 8)
    bias = D.uniform_f16(16, (N,))
    pre = u.astype(np.float64) * v.astype(np.float64) + bias.astype(np.float64)
    for la, lb in LAYOUTS:
        assert np.array_equal(run(lib, u, v, bias, la, lb, act=O.ACT_NONE), pre)
        assert np.array_equal(run(lib, u, v, bias, la, lb), np.maximum(pre, 0.0))


def pin_integer_exact(lib):
    """Entries in {-1,0,1}, bias in {-8..8}: every partial sum is a small
    integer, so the result equals numpy's exact integer matmul."""
    M, N, K = 23, 19, 37
    A, B, bias = D.random_problem(17, M, N, K, dist="int")
    ref = A.astype(np.int64) @ B.astype(np.int64) + bias.astype(np.int64)
    for la, lb in LAYOUTS:
        assert np.array_equal(run(lib, A, B, bias, la, lb, act=O.ACT_NONE), ref.astype(np.float64))
        assert np.array_equal(run(lib, A, B, bias, la, lb), np.maximum(ref, 0).astype(np.float64))


def pin_relu_invariant(lib):
    """ReLU output is >= 0, equals the pre-activation exactly where that is
    positive and is exactly 0 elsewhere; no-bias equals zero bias."""
    M, N, K = 17, 21, 40
    A, B, bias = D.random_problem(18, M, N, K)
    for la, lb in LAYOUTS:
        pre = run(lib, A, B, bias, la, lb, act=O.ACT_NONE)
        out = run(lib, A, B, bias, la, lb, act=O.ACT_RELU)
        assert (out >= 0).all()
        pos = pre > 0
        assert pos.any() and (~pos).any()
        assert np.array_equal(out[pos], pre[pos])
        assert (out[~pos] == 0).all()
        nob = run(lib, A, B, None, la, lb, act=O.ACT_NONE)
        zb = run(lib, A, B, np.zeros(N, np.float16), la, lb, act=O.ACT_NONE)
        assert np.array_equal(nob, zb)


def pin_brute_force_fraction(lib):
    """Tiny shapes in all layouts against exact rational arithmetic.  With
    K <= 8 and |values| <= 1 every product is a multiple of 2^-48 and every
    partial sum fits in 53 bits, so binary64 is exact and must agree."""
    rng = np.random.default_rng(19)
    for trial in range(12):
        M, N, K = (int(x) for x in rng.integers(1, 9, size=3))
        A, B, bias = D.random_problem(100 + trial, M, N, K)
        exact = [[sum((Fraction(float(A[i, k])) * Fraction(float(B[k, j])) for k in range(K)),
                      Fraction(0)) + Fraction(float(bias[j])) for j in range(N)] for i in range(M)]
        want_pre = np.array([[float(x) for x in r] for r in exact])
        want = np.array([[float(x) if x > 0 else 0.0 for x in r] for r in exact])
        for la, lb in LAYOUTS:
            assert np.array_equal(run(lib, A, B, bias, la, lb, act=O.ACT_NONE), want_pre)
            assert np.array_equal(run(lib, A, B, bias, la, lb), want)


def pin_numpy_matmul(lib):
    """Random 96 x 80 x 256 against numpy's float64 matmul (a library
    routine): relative error within a few binary64 ulps of the magnitude."""
    M, N, K = 96, 80, 256
    A, B, bias = D.random_problem(20, M, N, K)
    ref = A.astype(np.float64) @ B.astype(np.float64) + bias.astype(np.float64)
    scale = np.abs(A.astype(np.float64)) @ np.abs(B.astype(np.float64)) + 1.0
    for la, lb in LAYOUTS:
        got = run(lib, A, B, bias, la, lb, act=O.ACT_NONE)
        assert (np.abs(got - ref) <= 1e-12 * scale).all()


def pin_padded_leading_dims(lib):
    """Padded leading dimensions (NaN-filled padding) give the same result
    as packed storage, and row subsets match the full result."""
    M, N, K = 13, 11, 29
    A, B, bias = D.random_problem(21, M, N, K)
    for la, lb in LAYOUTS:
        packed = run(lib, A, B, bias, la, lb)
        padded = run(lib, A, B, bias, la, lb, pad=5)
        assert np.array_equal(packed, padded)
        rows = [12, 0, 7, 7]
        sub = run(lib, A, B, bias, la, lb, rows=rows)
        assert np.array_equal(sub, packed[rows])


def pin_degenerate(lib):
    """K = 0: the empty sum is 0, so out = relu(bias).  M or N = 0: empty."""
    N = 8
    bias = D.uniform_f16(22, (N,))
    A = np.zeros((3, 0), np.float16)
    B = np.zeros((0, N), np.float16)
    for la, lb in LAYOUTS:
        a_st = np.zeros((3, 1), np.float16) if la == D.ROW else np.zeros((1, 3), np.float16)
        b_st = np.zeros((1, N), np.float16) if lb == D.ROW else np.zeros((N, 1), np.float16)
        out = O.gemm_bias_act(a_st, la, b_st, lb, 3, N, 0, bias=bias, lda=a_st.shape[1],
                              ldb=b_st.shape[1], lib=lib)
        assert np.array_equal(out, np.broadcast_to(np.maximum(bias.astype(np.float64), 0), (3, N)))
    del A, B


PINS = [pin_decoder_all_patterns, pin_golden_worked_example, pin_all_ones, pin_identity,
        pin_rank1, pin_integer_exact, pin_relu_invariant, pin_brute_force_fraction,
        pin_numpy_matmul, pin_padded_leading_dims, pin_degenerate]

"""Pins for the oracle of the wider idioms (prologue ReLU, sum or difference
of two products, row or full bias added or subtracted, Sigmoid and Tanh).

Like oracle_pins.py: each ``pin_*`` takes an opened oracle library and
raises AssertionError when the library disagrees with a fact fixed by the
paper's listings or by mathematics -- a hand-derived worked example, exact
rational arithmetic, closed forms, identities between the activations, or
an independent library routine.
"""
import json
import os
from fractions import Fraction

import numpy as np
import scipy.special

from oracle import oracle as O
from paper_2006_12645_amd import datagen as D

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
LAYOUTS = [(D.ROW, D.ROW), (D.ROW, D.COL), (D.COL, D.ROW), (D.COL, D.COL)]
ACTS = {"none": O.ACT_NONE, "relu": O.ACT_RELU, "sigmoid": O.ACT_SIGMOID, "tanh": O.ACT_TANH}


def run(lib, A, B, la, lb, *, P=None, Q=None, second=0, pro=False, bias=None, bias_sign=1,
        act=O.ACT_NONE, pad=0, pad_pq=0, pad_bias=0, rows=None):
    """Store logical operands in the given layouts (optionally with padded
    leading dimensions; padding is NaN) and evaluate the fused oracle."""
    M, K = A.shape
    N = B.shape[1]
    a_st = D.store(A, la, (K if la == D.ROW else M) + pad)
    b_st = D.store(B, lb, (N if lb == D.ROW else K) + pad)
    p_st = q_st = None
    K2 = 0
    if second != 0:
        K2 = P.shape[1]
        p_st = D.store(P, la, (K2 if la == D.ROW else M) + pad_pq)
        q_st = D.store(Q, lb, (N if lb == D.ROW else K2) + pad_pq)
    bst = bias
    if bias is not None and bias.ndim == 2 and pad_bias:
        bst = D.store(bias, D.ROW, N + pad_bias)
    return O.fused(a_st, la, b_st, lb, M, N, K, prologue_relu=pro, second=second, p_store=p_st,
                   q_store=q_st, K2=K2, bias=bst, bias_sign=bias_sign, act=act, rows=rows,
                   nthreads=3, lib=lib)


def exact(A, B, P=None, Q=None, second=0, pro=False, bias=None, bias_sign=1):
    """Pre-activations in exact rational arithmetic."""
    def left(x):
        v = Fraction(float(x))
        return max(v, Fraction(0)) if pro else v
    M, K = A.shape
    N = B.shape[1]
    out = []
    for i in range(M):
        row = []
        for j in range(N):
            z = sum((left(A[i, k]) * Fraction(float(B[k, j])) for k in range(K)), Fraction(0))
            if second:
                r = sum((left(P[i, k]) * Fraction(float(Q[k, j])) for k in range(P.shape[1])),
                        Fraction(0))
                z = z + r if second > 0 else z - r
            if bias is not None:
                b = Fraction(float(bias[j] if bias.ndim == 1 else bias[i, j]))
                z = z + b if bias_sign > 0 else z - b
            row.append(z)
        out.append(row)
    return out


def pin_golden_listings_4_5(lib):
    """Hand-derived instance of Listings 4 and 5 (tests/golden), all layouts."""
    g = json.load(open(os.path.join(GOLDEN, "listing4_5_worked_example.json")))
    A, B = np.array(g["A"], np.float16), np.array(g["B"], np.float16)
    P, Q = np.array(g["P"], np.float16), np.array(g["Q"], np.float16)
    biases = {"none": None, "full": np.array(g["bias_full"], np.float16),
              "row": np.array(g["bias_row"], np.float16)}
    for case in g["cases"]:
        for la, lb in LAYOUTS:
            got = run(lib, A, B, la, lb, P=P, Q=Q, second=case["second"],
                      pro=case["prologue_relu"], bias=biases[case["bias"]],
                      bias_sign=case["bias_sign"], act=ACTS[case["act"]], pad=1, pad_pq=2,
                      pad_bias=1)
            assert np.array_equal(got, np.array(case["expected"], np.float64)), (case["name"], la, lb, got)


def pin_fused_brute_force(lib):
    """Tiny random instances of every combination against exact rational
    arithmetic.  K, K2 <= 8 and |values| <= 1 keep binary64 exact."""
    rng = np.random.default_rng(31)
    for trial in range(16):
        M, N, K, K2 = (int(x) for x in rng.integers(1, 9, size=4))
        A, B, _ = D.random_problem(300 + trial, M, N, K)
        P, Q, _ = D.random_problem(400 + trial, M, N, K2)
        second = (0, 1, -1)[trial % 3]
        pro = bool(trial & 1)
        bias = D.uniform_f16(500 + trial, (N,) if trial % 4 < 2 else (M, N))
        bias_sign = 1 if (trial >> 2) & 1 else -1
        ex = exact(A, B, P, Q, second, pro, bias, bias_sign)
        want = np.array([[float(x) for x in r] for r in ex])
        want_relu = np.array([[float(x) if x > 0 else 0.0 for x in r] for r in ex])
        for la, lb in LAYOUTS:
            kw = dict(P=P, Q=Q, second=second, pro=pro, bias=bias, bias_sign=bias_sign,
                      pad=trial % 3, pad_pq=(trial + 1) % 3, pad_bias=trial % 2)
            assert np.array_equal(run(lib, A, B, la, lb, act=O.ACT_NONE, **kw), want), (trial, la, lb)
            assert np.array_equal(run(lib, A, B, la, lb, act=O.ACT_RELU, **kw), want_relu), (trial, la, lb)


def pin_prologue_closed_forms(lib):
    """relu on a non-positive A leaves only the bias; with A(i,k) = +-1 by
    the parity of k and B = 1, relu(A).B counts the positive entries."""
    M, N, K = 6, 5, 13
    neg = -np.abs(D.uniform_f16(32, (M, K)))
    B = D.uniform_f16(33, (K, N))
    bias = D.uniform_f16(34, (N,))
    alt = np.array([[1.0 if k % 2 == 0 else -1.0 for k in range(K)] for _ in range(M)], np.float16)
    ones = np.ones((K, N), np.float16)
    for la, lb in LAYOUTS:
        got = run(lib, neg, B, la, lb, pro=True, bias=bias, act=O.ACT_NONE)
        assert np.array_equal(got, np.broadcast_to(bias.astype(np.float64), (M, N)))
        got = run(lib, alt, ones, la, lb, pro=True)
        assert (got == (K + 1) // 2).all(), got
        got = run(lib, alt, ones, la, lb, pro=False)
        assert (got == K % 2).all(), got


def pin_second_product_identities(lib):
    """P.Q = A.B cancels exactly under subtract and doubles under add
    (checked against numpy's matmul); K2 != K against numpy as well."""
    M, N, K = 9, 12, 40
    A, B, bias = D.random_problem(35, M, N, K)
    ref = A.astype(np.float64) @ B.astype(np.float64)
    scale = np.abs(A.astype(np.float64)) @ np.abs(B.astype(np.float64)) + 1.0
    P2, Q2, _ = D.random_problem(36, M, N, 300)
    ref2 = P2.astype(np.float64) @ Q2.astype(np.float64)
    scale2 = np.abs(P2.astype(np.float64)) @ np.abs(Q2.astype(np.float64)) + 1.0
    for la, lb in LAYOUTS:
        got = run(lib, A, B, la, lb, P=A, Q=B, second=-1, bias=bias, act=O.ACT_NONE)
        assert np.array_equal(got, np.broadcast_to(bias.astype(np.float64), (M, N)))
        got = run(lib, A, B, la, lb, P=A, Q=B, second=1, act=O.ACT_NONE)
        assert (np.abs(got - 2 * ref) <= 1e-12 * scale).all()
        got = run(lib, A, B, la, lb, P=P2, Q=Q2, second=1, act=O.ACT_NONE, pad_pq=3)
        assert (np.abs(got - (ref + ref2)) <= 1e-12 * (scale + scale2)).all()
        got = run(lib, A, B, la, lb, P=P2, Q=Q2, second=-1, act=O.ACT_NONE, pad_pq=3)
        assert (np.abs(got - (ref - ref2)) <= 1e-12 * (scale + scale2)).all()


def pin_full_bias_indexing(lib):
    """With K = 0 (empty sums) the output is the bias tile itself, indexed
    bias[i*ldbias + j] through a padded leading dimension; subtracting it
    negates it; a row subset picks the matching bias rows."""
    M, N = 7, 6
    bias = D.uniform_f16(37, (M, N), -4, 4)
    A = np.zeros((M, 0), np.float16)
    B = np.zeros((0, N), np.float16)
    want = bias.astype(np.float64)
    for la, lb in LAYOUTS:
        got = run(lib, A, B, la, lb, bias=bias, pad=1, pad_bias=3)
        assert np.array_equal(got, want)
        got = run(lib, A, B, la, lb, bias=bias, bias_sign=-1, pad=1, pad_bias=3)
        assert np.array_equal(got, -want)
        got = run(lib, A, B, la, lb, bias=bias, pad=1, pad_bias=3, rows=[6, 1, 1])
        assert np.array_equal(got, want[[6, 1, 1]])


def pin_activations_closed_forms(lib):
    """sigmoid(0) = 1/2 and tanh(0) = 0 exactly; far from 0 both saturate to
    their limits; sigmoid(x) + sigmoid(-x) = 1; tanh is odd; and
    tanh(x) = 2 sigmoid(2x) - 1 ties the two routines together (doubling B
    and the bias doubles the pre-activation exactly)."""
    M, N = 3, 4
    zeroA = np.zeros((M, 0), np.float16)
    zeroB = np.zeros((0, N), np.float16)
    for la, lb in LAYOUTS:
        assert (run(lib, zeroA, zeroB, la, lb, act=O.ACT_SIGMOID) == 0.5).all()
        assert (run(lib, zeroA, zeroB, la, lb, act=O.ACT_TANH) == 0.0).all()
        far = np.full((N,), -40.0, np.float16)
        s = run(lib, zeroA, zeroB, la, lb, bias=far, act=O.ACT_SIGMOID)
        assert (s > 0).all() and (s < 1e-17).all()
        t = run(lib, zeroA, zeroB, la, lb, bias=far, act=O.ACT_TANH)
        assert (t == -1.0).all()
    M, N, K = 11, 9, 24
    A, B, bias = D.random_problem(38, M, N, K)
    for la, lb in LAYOUTS:
        sp = run(lib, A, B, la, lb, bias=bias, act=O.ACT_SIGMOID)
        sn = run(lib, A, -B, la, lb, bias=-bias, act=O.ACT_SIGMOID)
        assert np.allclose(sp + sn, 1.0, rtol=0, atol=4e-16)
        assert ((sp > 0) & (sp < 1)).all()
        tp = run(lib, A, B, la, lb, bias=bias, act=O.ACT_TANH)
        tn = run(lib, A, -B, la, lb, bias=-bias, act=O.ACT_TANH)
        assert np.array_equal(tp, -tn)
        s2 = run(lib, A, 2 * B, la, lb, bias=2 * bias, act=O.ACT_SIGMOID)
        assert np.allclose(tp, 2 * s2 - 1, rtol=0, atol=1e-15)
        # monotone in the pre-activation
        pre = run(lib, A, B, la, lb, bias=bias, act=O.ACT_NONE)
        order = np.argsort(pre, axis=None)
        assert (np.diff(sp.ravel()[order]) >= 0).all() and (np.diff(tp.ravel()[order]) >= 0).all()


def pin_activations_vs_library(lib):
    """Sigmoid and Tanh of the oracle's own pre-activations against scipy's
    expit and numpy's tanh (independent implementations), to 2 ulps."""
    M, N, K = 40, 33, 64
    A, B, bias = D.random_problem(39, M, N, K)
    for la, lb in [(D.ROW, D.COL), (D.COL, D.ROW)]:
        pre = run(lib, A, B, la, lb, bias=bias, act=O.ACT_NONE, pro=True)
        s = run(lib, A, B, la, lb, bias=bias, act=O.ACT_SIGMOID, pro=True)
        t = run(lib, A, B, la, lb, bias=bias, act=O.ACT_TANH, pro=True)
        r = run(lib, A, B, la, lb, bias=bias, act=O.ACT_RELU, pro=True)
        assert np.allclose(s, scipy.special.expit(pre), rtol=4.5e-16, atol=1e-300)
        assert np.allclose(t, np.tanh(pre), rtol=4.5e-16, atol=1e-300)
        assert np.array_equal(r, np.where(pre > 0, pre, 0.0))


PINS = [pin_golden_listings_4_5, pin_fused_brute_force, pin_prologue_closed_forms,
        pin_second_product_identities, pin_full_bias_indexing, pin_activations_closed_forms,
        pin_activations_vs_library]

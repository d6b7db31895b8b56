"""ctypes front end of the C oracle (oracle_gba.c).

Test infrastructure only: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg, never by the HIP library or its binding.

Arrays are numpy: fp16 operands are passed as their raw bit patterns, the
result comes back as float64.  See oracle_gba.c for the definition computed
(the Problem Statement section's matmul followed by the ReLU-of-add
statement, and the prologue / sum-of-matmuls / other-pointwise-op idioms,
evaluated in binary64 with k ascending).
"""
import ctypes
import os

import numpy as np

from . import build_oracle

ROW, COL = 0, 1
ACT_NONE, ACT_RELU, ACT_SIGMOID, ACT_TANH = 0, 1, 2, 3
BIAS_NONE, BIAS_ROW, BIAS_FULL = 0, 1, 2

_lib = None


def load_library(path):
    """Open a compiled oracle library and declare its entry points."""
    lib = ctypes.CDLL(path)
    i64, vp = ctypes.c_int64, ctypes.c_void_p
    lib.oracle_f16_to_f64.restype = ctypes.c_double
    lib.oracle_f16_to_f64.argtypes = [ctypes.c_uint16]
    lib.oracle_round_f16.restype = ctypes.c_double
    lib.oracle_round_f16.argtypes = [ctypes.c_double]
    lib.oracle_gemm_bias_act_rows_f64.restype = ctypes.c_int
    lib.oracle_gemm_bias_act_rows_f64.argtypes = [
        ctypes.c_int, ctypes.c_int, i64, i64, i64, vp, i64, vp, i64, vp,
        ctypes.c_int, vp, i64, vp, i64, ctypes.c_int]
    ci = ctypes.c_int
    lib.oracle_fused_rows_f64.restype = ci
    lib.oracle_fused_rows_f64.argtypes = [
        ci, ci, i64, i64, i64, vp, i64, vp, i64,          # layouts, M N K, A lda, B ldb
        ci, ci, i64, vp, i64, vp, i64,                    # pro_relu, second, K2, P ldp, Q ldq
        ci, ci, vp, i64, ci, ci,                          # bias kind/sign, bias ldbias, act, acc16
        vp, i64, vp, i64, ci]                             # rows nrows, out ldo, nthreads
    return lib


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(build_oracle.LIB):
            build_oracle.build()
        _lib = load_library(build_oracle.LIB)
    return _lib


def default_threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(n, 16))


def f16_to_f64(bits: int, lib=None) -> float:
    """Decode one fp16 bit pattern with the oracle's own decoder."""
    return (lib or _load()).oracle_f16_to_f64(int(bits) & 0xFFFF)


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _as_bits(x):
    if x is None:
        return None
    x = np.ascontiguousarray(x)
    if x.dtype == np.float16:
        x = x.view(np.uint16)
    if x.dtype != np.uint16:
        raise TypeError("oracle operands must be float16 or uint16 bit patterns")
    return x


def gemm_bias_act(a_store, layout_a, b_store, layout_b, M, N, K, bias=None,
                  act=ACT_RELU, lda=None, ldb=None, rows=None, nthreads=None, lib=None):
    """Oracle result as float64, shape (len(rows) or M, N).

    ``a_store``/``b_store`` are the stored 2-D fp16 arrays: for a row-major
    A it is M x lda, for a column-major A it is K x lda (so A(i,k) is
    a_store[k, i]); likewise B is K x ldb row-major or N x ldb column-major.
    """
    lib = lib or _load()
    a = _as_bits(a_store)
    b = _as_bits(b_store)
    bi = _as_bits(bias)
    if lda is None:
        lda = a.shape[1] if a.ndim == 2 else (K if layout_a == ROW else M)
    if ldb is None:
        ldb = b.shape[1] if b.ndim == 2 else (N if layout_b == ROW else K)
    if rows is None:
        r = None
        nrows = M
    else:
        r = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
        nrows = r.shape[0]
    out = np.zeros((nrows, N), dtype=np.float64)
    rc = lib.oracle_gemm_bias_act_rows_f64(
        int(layout_a), int(layout_b), int(M), int(N), int(K), _ptr(a), int(lda), _ptr(b), int(ldb),
        _ptr(bi), int(act), _ptr(r), int(nrows), _ptr(out), int(max(N, 1)),
        int(nthreads or default_threads()))
    if rc != 0:
        raise ValueError(f"oracle rejected the arguments (rc={rc})")
    return out


def round_f16(x: float, lib=None) -> float:
    """The oracle's binary64 -> binary16 rounding (ties to even)."""
    return (lib or _load()).oracle_round_f16(float(x))


def _ld(store, default):
    return store.shape[1] if store is not None and store.ndim == 2 else default


def fused(a_store, layout_a, b_store, layout_b, M, N, K, *, prologue_relu=False,
          second=0, p_store=None, q_store=None, K2=0, bias=None, bias_kind=None,
          bias_sign=1, act=ACT_RELU, lda=None, ldb=None, ldp=None, ldq=None, ldbias=None,
          acc16=False, rows=None, nthreads=None, lib=None):
    """Oracle of the general fused operation as float64, shape (len(rows) or M, N).

    ``second`` is 0 (one product), +1 (add P.Q) or -1 (subtract P.Q); P and
    Q are stored like A and B.  ``bias`` is a length-N vector (bias_kind
    BIAS_ROW, the default for a 1-D bias) or an M x ldbias array (BIAS_FULL,
    the default for a 2-D bias); ``bias_sign`` -1 subtracts it.  ``acc16``
    evaluates the fp16-accumulation reading (running sum rounded to binary16
    after every aligned group of 32 k of each product) instead of the exact
    binary64 sums.
    """
    lib = lib or _load()
    a, b = _as_bits(a_store), _as_bits(b_store)
    pp, qq = _as_bits(p_store), _as_bits(q_store)
    bi = _as_bits(bias)
    if bias_kind is None:
        bias_kind = BIAS_NONE if bi is None else (BIAS_ROW if bi.ndim == 1 else BIAS_FULL)
    if ldbias is None:
        ldbias = bi.shape[1] if bi is not None and bi.ndim == 2 else N
    lda = lda if lda is not None else _ld(a, K if layout_a == ROW else M)
    ldb = ldb if ldb is not None else _ld(b, N if layout_b == ROW else K)
    ldp = ldp if ldp is not None else _ld(pp, K2 if layout_a == ROW else M)
    ldq = ldq if ldq is not None else _ld(qq, N if layout_b == ROW else K2)
    if rows is None:
        r, nrows = None, M
    else:
        r = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
        nrows = r.shape[0]
    out = np.zeros((nrows, N), dtype=np.float64)
    rc = lib.oracle_fused_rows_f64(
        int(layout_a), int(layout_b), int(M), int(N), int(K), _ptr(a), int(lda), _ptr(b), int(ldb),
        int(bool(prologue_relu)), int(second), int(K2), _ptr(pp), int(ldp), _ptr(qq), int(ldq),
        int(bias_kind), int(bias_sign), _ptr(bi), int(ldbias), int(act), int(bool(acc16)),
        _ptr(r), int(nrows), _ptr(out), int(max(N, 1)), int(nthreads or default_threads()))
    if rc != 0:
        raise ValueError(f"oracle rejected the arguments (rc={rc})")
    return out

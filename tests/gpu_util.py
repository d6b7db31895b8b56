"""Helpers shared by the GPU tests: device copies of stored operands and the
element-wise parity check against the oracle."""
import numpy as np

from oracle import oracle as O
from paper_2006_12645_amd import datagen as D

# |gpu - oracle| <= ATOL + RTOL * |oracle|: fp32 accumulation uses the bound
# the method is held to; fp16 accumulation (running sum rounded to fp16 every
# 32 k) the looser stated one.
TOL = {"f32": (1e-2, 1e-2), "f16": (5e-2, 5e-2)}


def device_operand(logical, layout, pad=0):
    """A CUDA tensor of logical shape rows x cols stored in the given layout
    with leading dimension extent + pad (a strided view into the storage)."""
    import torch
    rows, cols = logical.shape
    ext = cols if layout == D.ROW else rows
    st = D.store(logical, layout, ext + pad)
    t = torch.from_numpy(st).cuda()
    if layout == D.ROW:
        return t[:, :cols]
    return t[:, :rows].t()


def oracle_for(A, B, bias, act=O.ACT_RELU, rows=None):
    """Oracle result for logical A, B (stored RC, the layout does not change
    the definition)."""
    M, K = A.shape
    N = B.shape[1]
    return O.gemm_bias_act(D.store(A, D.ROW), D.ROW, D.store(B, D.COL), D.COL, M, N, K,
                           bias=bias, act=act, rows=rows)


def assert_close(gpu_f16, ref, accum="f32", what=""):
    g = np.asarray(gpu_f16, dtype=np.float64)
    atol, rtol = TOL[accum]
    if g.shape != np.shape(ref):
        raise AssertionError(f"{what}: shape {g.shape} against the oracle's {np.shape(ref)}")
    err = np.abs(g - ref)
    bound = atol + rtol * np.abs(ref)
    # written as "not within" so that a NaN or infinite output (for which
    # every comparison is false) counts as a mismatch
    bad = ~(err <= bound)
    if bad.any():
        idx = np.argwhere(bad)[:5]
        raise AssertionError(
            f"{what}: {int(bad.sum())} of {bad.size} outside |d| <= {atol} + {rtol}|ref|; "
            f"max err {np.nanmax(np.where(np.isfinite(err), err, np.inf)):.4g}; first at {idx.tolist()}: "
            f"gpu {g[tuple(idx[0])]} ref {ref[tuple(idx[0])]}")
    return float(err.max())

"""ctypes binding of libgba.so (C ABI in include/gba.h).

Argument marshalling only: every step of the computation runs in the HIP
library.  torch supplies device memory and the stream; this module reads
tensor pointers, strides and the current stream and forwards them.  If the
library has not been built, importing the entry points raises -- there is no
fallback implementation.
"""
import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libgba.so")

GBA_ROW_MAJOR, GBA_COL_MAJOR = 0, 1
GBA_ACT_NONE, GBA_ACT_RELU = 0, 1
GBA_ACC_F32, GBA_ACC_F16 = 0, 1
GBA_OK, GBA_EINVAL, GBA_EUNSUPPORTED, GBA_EHIP = 0, 1, 2, 3

ACTS = {"none": GBA_ACT_NONE, "relu": GBA_ACT_RELU}
ACCS = {"f32": GBA_ACC_F32, "fp32": GBA_ACC_F32, "f16": GBA_ACC_F16, "fp16": GBA_ACC_F16}

# Every function include/gba.h declares, with its ctypes signature.
_i64, _int, _vp, _cp = ctypes.c_int64, ctypes.c_int, ctypes.c_void_p, ctypes.c_char_p
_GEMM_ARGS = [_int, _int, _i64, _i64, _i64, _vp, _i64, _vp, _i64, _vp, _vp, _i64, _int, _int]
SIGNATURES = {
    "gemm_bias_act": (_int, _GEMM_ARGS + [_vp]),
    "gemm_bias_act_tile": (_int, _GEMM_ARGS + [_int, _vp]),
    "gba_num_tiles": (_int, []),
    "gba_tile_info": (_int, [_int] + [ctypes.POINTER(_int)] * 5),
    "gba_select_tile": (_int, [_int, _int, _i64, _i64, _i64, _int]),
    "gba_bias_add_f16": (_int, [_i64, _i64, _vp, _i64, _vp, _vp]),
    "gba_relu_f16": (_int, [_i64, _i64, _vp, _i64, _vp]),
    "gba_status_string": (_cp, [_int]),
    "gba_version": (_cp, []),
}

_lib = None


class GbaError(RuntimeError):
    def __init__(self, status, what):
        self.status = status
        super().__init__(f"{what}: {lib().gba_status_string(status).decode()}")


def lib():
    """The loaded library (loaded once).  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -c 'import __graft_entry__ as g; g.build()'`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _check(status, what):
    if status != GBA_OK:
        raise GbaError(status, what)


def _stream_handle(stream, device):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream(device)
    return ctypes.c_void_p(stream.cuda_stream)


def operand_layout(t, rows, cols):
    """(layout, ld) of a 2-D tensor holding a logical rows x cols matrix."""
    if t.dim() != 2 or tuple(t.shape) != (rows, cols):
        raise ValueError(f"expected a {rows}x{cols} matrix, got shape {tuple(t.shape)}")
    s0, s1 = t.stride()
    if (s1 == 1 or cols <= 1) and (rows <= 1 or s0 >= cols):
        return GBA_ROW_MAJOR, (s0 if rows > 1 else max(cols, 1))
    if (s0 == 1 or rows <= 1) and (cols <= 1 or s1 >= rows):
        return GBA_COL_MAJOR, (s1 if cols > 1 else max(rows, 1))
    raise ValueError("operand must be row- or column-major (one unit stride)")


def _row_major_ld(t, what):
    M, N = t.shape
    if M > 1 and (N > 1 and t.stride(1) != 1 or t.stride(0) < N):
        raise ValueError(f"{what} must be a row-major (M, N) matrix")
    return t.stride(0) if M > 1 else max(N, 1)


def gemm_bias_act(A, B, bias=None, act="relu", accum="f32", out=None, tile=None, stream=None):
    """out = act(A @ B + bias) in one fused kernel.

    A: (M, K) fp16 CUDA tensor, row- or column-major (any leading dimension).
    B: (K, N) fp16 CUDA tensor, row- or column-major.
    bias: (N,) fp16 contiguous tensor or None.  out: (M, N) row-major fp16
    (allocated when None).  tile: force a tile configuration id.
    """
    import torch
    M, K = A.shape
    K2, N = B.shape
    if K2 != K:
        raise ValueError("inner dimensions differ")
    for name, t in (("A", A), ("B", B), ("bias", bias), ("out", out)):
        if t is not None and (t.dtype != torch.float16 or not t.is_cuda):
            raise TypeError(f"{name} must be a float16 CUDA tensor")
    la, lda = operand_layout(A, M, K)
    lb, ldb = operand_layout(B, K, N)
    if bias is not None and (bias.dim() != 1 or bias.shape[0] != N or
                             (N > 1 and bias.stride(0) != 1)):
        raise ValueError("bias must be a contiguous (N,) vector")
    if out is None:
        out = torch.empty((M, N), dtype=torch.float16, device=A.device)
    if out.dim() != 2 or tuple(out.shape) != (M, N):
        raise ValueError("out must be an (M, N) matrix")
    ldc = _row_major_ld(out, "out")
    args = [la, lb, M, N, K, A.data_ptr(), lda, B.data_ptr(), ldb,
            None if bias is None else bias.data_ptr(), out.data_ptr(), ldc,
            ACTS[act], ACCS[accum]]
    s = _stream_handle(stream, A.device)
    if tile is None:
        _check(lib().gemm_bias_act(*args, s), "gemm_bias_act")
    else:
        _check(lib().gemm_bias_act_tile(*args, int(tile), s), "gemm_bias_act_tile")
    return out


def bias_add_(C, bias, stream=None):
    """In place: C = fp16(C + bias[None, :]) (unfused baseline piece)."""
    M, N = C.shape
    ldc = _row_major_ld(C, "C")
    _check(lib().gba_bias_add_f16(M, N, C.data_ptr(), ldc, bias.data_ptr(),
                                  _stream_handle(stream, C.device)), "gba_bias_add_f16")
    return C


def relu_(C, stream=None):
    """In place: C = max(C, 0) (unfused baseline piece)."""
    M, N = C.shape
    ldc = _row_major_ld(C, "C")
    _check(lib().gba_relu_f16(M, N, C.data_ptr(), ldc, _stream_handle(stream, C.device)),
           "gba_relu_f16")
    return C


def unfused_gemm_bias_relu(A, B, bias, out=None, tile=None, stream=None):
    """The three-launch baseline chain: GEMM (no epilogue), bias add, ReLU."""
    out = gemm_bias_act(A, B, None, act="none", out=out, tile=tile, stream=stream)
    bias_add_(out, bias, stream)
    relu_(out, stream)
    return out


def num_tiles():
    return lib().gba_num_tiles()


def tile_info(tile_id):
    vals = [ctypes.c_int() for _ in range(5)]
    _check(lib().gba_tile_info(int(tile_id), *[ctypes.byref(v) for v in vals]), "gba_tile_info")
    return dict(zip(("bm", "bn", "bk", "waves", "split_k"), (v.value for v in vals)))


def select_tile(M, N, K, layout_a=GBA_ROW_MAJOR, layout_b=GBA_COL_MAJOR, accum="f32"):
    return lib().gba_select_tile(layout_a, layout_b, M, N, K, ACCS[accum])


def version():
    return lib().gba_version().decode()

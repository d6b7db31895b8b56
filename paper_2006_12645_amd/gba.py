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
GBA_ACT_NONE, GBA_ACT_RELU, GBA_ACT_SIGMOID, GBA_ACT_TANH = 0, 1, 2, 3
GBA_ACC_F32, GBA_ACC_F16 = 0, 1
GBA_OK, GBA_EINVAL, GBA_EUNSUPPORTED, GBA_EHIP, GBA_ESCRATCH = 0, 1, 2, 3, 4
GBA_NOALLOC_SCRATCH_BYTES = 16 << 20
GBA_PRO_NONE, GBA_PRO_RELU = 0, 1
GBA_SECOND_NONE, GBA_SECOND_ADD, GBA_SECOND_SUB = 0, 1, 2
GBA_BIAS_NONE, GBA_BIAS_ROW, GBA_BIAS_FULL = 0, 1, 2
GBA_OP_ADD, GBA_OP_SUB = 0, 1

ACTS = {"none": GBA_ACT_NONE, "relu": GBA_ACT_RELU, "sigmoid": GBA_ACT_SIGMOID,
        "tanh": GBA_ACT_TANH}
ACCS = {"f32": GBA_ACC_F32, "fp32": GBA_ACC_F32, "f16": GBA_ACC_F16, "fp16": GBA_ACC_F16}
OPS = {"add": GBA_OP_ADD, "sub": GBA_OP_SUB}

_i64, _int, _vp, _cp = ctypes.c_int64, ctypes.c_int, ctypes.c_void_p, ctypes.c_char_p


class FusedDesc(ctypes.Structure):
    """Mirror of struct gba_fused_desc (C enums are int)."""
    _fields_ = [("layoutA", _int), ("layoutB", _int), ("M", _i64), ("N", _i64), ("K", _i64),
                ("A", _vp), ("lda", _i64), ("B", _vp), ("ldb", _i64),
                ("prologue", _int), ("second", _int), ("K2", _i64),
                ("P", _vp), ("ldp", _i64), ("Q", _vp), ("ldq", _i64),
                ("bias_kind", _int), ("bias_op", _int), ("bias", _vp), ("ldbias", _i64),
                ("act", _int), ("accum", _int), ("C", _vp), ("ldc", _i64), ("tile_id", _int),
                ("split_k", _int), ("workspace", _vp), ("workspace_bytes", ctypes.c_size_t)]


# Every function include/gba.h declares, with its ctypes signature.
_GEMM_ARGS = [_int, _int, _i64, _i64, _i64, _vp, _i64, _vp, _i64, _vp, _vp, _i64, _int, _int]
SIGNATURES = {
    "gemm_bias_act": (_int, _GEMM_ARGS + [_vp]),
    "gemm_bias_act_tile": (_int, _GEMM_ARGS + [_int, _vp]),
    "gba_num_tiles": (_int, []),
    "gba_tile_info": (_int, [_int] + [ctypes.POINTER(_int)] * 5),
    "gba_select_tile": (_int, [_int, _int, _i64, _i64, _i64, _int]),
    "gba_bias_add_f16": (_int, [_i64, _i64, _vp, _i64, _vp, _vp]),
    "gba_relu_f16": (_int, [_i64, _i64, _vp, _i64, _vp]),
    "gba_bias_act_f16": (_int, [_i64, _i64, _vp, _i64, _vp, _int, _vp]),
    "gba_add_f16": (_int, [_i64, _i64, _vp, _i64, _vp, _i64, _vp]),
    "gba_fused_desc_init": (None, [ctypes.POINTER(FusedDesc)]),
    "gba_fused_gemm": (_int, [ctypes.POINTER(FusedDesc), _vp]),
    "gba_fused_gemm_noalloc": (_int, [ctypes.POINTER(FusedDesc), _vp]),
    "gba_fused_workspace_size": (_int, [ctypes.POINTER(FusedDesc), ctypes.POINTER(ctypes.c_size_t)]),
    "gba_fused_tile": (_int, [ctypes.POINTER(FusedDesc), ctypes.POINTER(_int)]),
    "gba_status_string": (_cp, [_int]),
    "gba_version": (_cp, []),
}

_lib = None


class GbaError(RuntimeError):
    def __init__(self, status, what):
        self.status = status
        super().__init__(f"{what}: {lib().gba_status_string(status).decode()}")


def lib():
    """The loaded library (loaded once).  Raises if it has not been built.

    torch is imported first: its wheel carries its own HIP runtime, which
    the library then binds to (both name it libamdhip64.so.7).  Loaded
    before torch, the library would bring in the system's runtime and torch
    its own beside it: two runtimes in one process, and a launch on one of
    torch's streams fails."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -c 'import __graft_entry__ as g; g.build()'`")
        import torch  # noqa: F401  (load order: see above)
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
    """The HIP stream to launch on: `stream`, else torch's current stream of
    `device` (read through torch's raw-pointer accessor when it has one,
    which costs ~0.1 us against ~2 us for a Stream object)."""
    import torch
    if stream is None:
        raw = getattr(torch._C, "_cuda_getCurrentRawStream", None)
        dev = torch.device(device) if device is not None else torch.device("cuda")
        if raw is not None:
            return ctypes.c_void_p(raw(dev.index if dev.index is not None else torch.cuda.current_device()))
        stream = torch.cuda.current_stream(dev)
    return ctypes.c_void_p(stream.cuda_stream)


def _stored_as(t, rows, cols, layout):
    """Whether a 2-D tensor holding a logical rows x cols matrix can be
    passed in `layout` (a single row or column fits either layout)."""
    s0, s1 = t.stride()
    if layout == GBA_ROW_MAJOR:
        return (s1 == 1 or cols <= 1) and (rows <= 1 or s0 >= cols)
    return (s0 == 1 or rows <= 1) and (cols <= 1 or s1 >= rows)


def operand_layout(t, rows, cols, want=None):
    """(layout, ld) of a 2-D tensor holding a logical rows x cols matrix;
    ``want`` asks for that layout (for operands that must match another)."""
    if t.dim() != 2 or tuple(t.shape) != (rows, cols):
        raise ValueError(f"expected a {rows}x{cols} matrix, got shape {tuple(t.shape)}")
    s0, s1 = t.stride()
    if want in (None, GBA_ROW_MAJOR) and _stored_as(t, rows, cols, GBA_ROW_MAJOR):
        return GBA_ROW_MAJOR, (s0 if rows > 1 else max(cols, 1))
    if want in (None, GBA_COL_MAJOR) and _stored_as(t, rows, cols, GBA_COL_MAJOR):
        return GBA_COL_MAJOR, (s1 if cols > 1 else max(rows, 1))
    if want is not None:
        raise ValueError("P and Q must be stored in the layouts of A and B")
    raise ValueError("operand must be row- or column-major (one unit stride)")


def shared_layout(x, rows, cols, y, rows2, cols2):
    """The layout two operands that must share one (A and P, or B and Q)
    are passed in: row-major if both can be, else column-major.  An operand
    with a single row or column fits either, so the other one decides."""
    for t, r, c in ((x, rows, cols), (y, rows2, cols2)):
        if t.dim() != 2 or tuple(t.shape) != (r, c):
            raise ValueError(f"expected a {r}x{c} matrix, got shape {tuple(t.shape)}")
    for layout in (GBA_ROW_MAJOR, GBA_COL_MAJOR):
        if _stored_as(x, rows, cols, layout) and _stored_as(y, rows2, cols2, layout):
            return layout
    raise ValueError("P and Q must be stored in the layouts of A and B")


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


def new_desc():
    """A FusedDesc holding the library's defaults (gba_fused_desc_init)."""
    d = FusedDesc()
    lib().gba_fused_desc_init(ctypes.byref(d))
    return d


def fused_gemm_desc(desc, stream=None, device=None):
    """Launch gba_fused_gemm on a filled FusedDesc (raises on error)."""
    _check(lib().gba_fused_gemm(ctypes.byref(desc), _stream_handle(stream, device)), "gba_fused_gemm")


def fused_gemm_desc_noalloc(desc, stream=None, device=None):
    """Launch gba_fused_gemm_noalloc on a filled FusedDesc: a split reduction
    uses the library's static scratch, nothing is allocated (raises on
    error)."""
    _check(lib().gba_fused_gemm_noalloc(ctypes.byref(desc), _stream_handle(stream, device)),
           "gba_fused_gemm_noalloc")


def workspace_size(desc):
    """Bytes of workspace a filled FusedDesc would use to split its reduction."""
    n = ctypes.c_size_t(0)
    _check(lib().gba_fused_workspace_size(ctypes.byref(desc), ctypes.byref(n)), "gba_fused_workspace_size")
    return n.value


def fused_tile(desc):
    """Tile id a filled FusedDesc would run on (-1: general path)."""
    t = _int(-1)
    _check(lib().gba_fused_tile(ctypes.byref(desc), ctypes.byref(t)), "gba_fused_tile")
    return t.value


# Zero-filled workspaces, one per (device, stream): the library leaves every
# byte a call used at zero when the call completes, so a workspace stays
# ready for the next call in that stream's order.  A workspace that is replaced by
# a larger one is kept alive (in _retired), since a graph captured earlier
# may still hold its address.
_workspaces = {}
_retired = []


def stream_capturing(stream):
    """True while `stream` is being captured into a HIP graph."""
    import torch
    with torch.cuda.stream(stream):
        return torch.cuda.is_current_stream_capturing()


def stream_workspace(nbytes, device, stream=None):
    """A zero-filled uint8 CUDA tensor of at least nbytes for calls on `stream`.

    Allocating and zero-filling it is itself GPU work on `stream`, so it is
    refused while the stream is being captured into a graph: make one eager
    call first (the cached workspace is then reused during capture), or pass
    a caller-owned zero-filled workspace.
    """
    import torch
    if stream is None:
        stream = torch.cuda.current_stream(device)
    key = (torch.device(device).index, stream.cuda_stream)
    ws = _workspaces.get(key)
    if ws is None or ws.numel() < nbytes:
        if stream_capturing(stream):
            raise RuntimeError(
                f"workspace='auto' would allocate and zero-fill {nbytes} bytes while the stream is "
                "being captured into a graph; pass a zero-filled uint8 CUDA tensor of at least that "
                "size as `workspace`, or make one call before the capture")
        if ws is not None:
            _retired.append(ws)
        with torch.cuda.stream(stream):
            ws = torch.zeros(max(nbytes, 1 << 20), dtype=torch.uint8, device=device)
        _workspaces[key] = ws
    return ws


def fused_gemm(A, B, *, P=None, Q=None, second="add", prologue=None, bias=None, bias_op="add",
               act="relu", accum="f32", out=None, tile=None, split=None, workspace="auto",
               stream=None):
    """out = act((pro(A) @ B  +/-  pro(P) @ Q)  +/-  bias) in one kernel.

    A (M, K), B (K, N): fp16 CUDA tensors, row- or column-major.  P (M, K2)
    and Q (K2, N), if given, must use the layouts of A and B; ``second`` is
    "add" or "sub".  prologue: None or "relu" (applied to A and P).  bias:
    None, an (N,) vector or a row-major (M, N) matrix; ``bias_op`` "add" or
    "sub".  act: "none", "relu", "sigmoid", "tanh".  out: (M, N) row-major
    fp16, allocated when None.  split: None (library's choice) or the number
    of workgroups each output tile's reduction is split across (1: never).
    workspace: "auto" (a cached zero-filled buffer for this stream), None
    (no split), a zero-filled uint8 CUDA tensor owned by the caller, or
    "static" (gba_fused_gemm_noalloc: the library's own static scratch,
    nothing allocated).
    """
    import torch
    M, K = A.shape
    Kb, N = B.shape
    if Kb != K:
        raise ValueError("inner dimensions of A and B differ")
    if (P is None) != (Q is None):
        raise ValueError("P and Q come together")
    for name, t in (("A", A), ("B", B), ("P", P), ("Q", Q), ("bias", bias), ("out", out)):
        if t is not None and (t.dtype != torch.float16 or not t.is_cuda):
            raise TypeError(f"{name} must be a float16 CUDA tensor")
    d = new_desc()
    d.M, d.N, d.K = M, N, K
    d.A, d.B = A.data_ptr(), B.data_ptr()
    d.prologue = {None: GBA_PRO_NONE, "none": GBA_PRO_NONE, "relu": GBA_PRO_RELU}[prologue]
    K2 = 0
    if P is not None:
        Mp, K2 = P.shape
        K2q, Nq = Q.shape
        if Mp != M or Nq != N or K2q != K2:
            raise ValueError("P @ Q must be an (M, N) product")
        d.second = {"add": GBA_SECOND_ADD, "sub": GBA_SECOND_SUB}[second]
        d.K2, d.P, d.Q = K2, P.data_ptr(), Q.data_ptr()
    # Layouts come from the operands that are read; an empty reduction's
    # operands are never read, so their layout and leading dimension are
    # free (the smallest legal ones are passed).
    want_a = want_b = None
    if K > 0 and K2 > 0:
        want_a, want_b = shared_layout(A, M, K, P, M, K2), shared_layout(B, K, N, Q, K2, N)
    if K > 0:
        d.layoutA, d.lda = operand_layout(A, M, K, want=want_a)
        d.layoutB, d.ldb = operand_layout(B, K, N, want=want_b)
    if K2 > 0:
        d.layoutA, d.ldp = operand_layout(P, M, K2, want=want_a)
        d.layoutB, d.ldq = operand_layout(Q, K2, N, want=want_b)
    row_a, row_b = d.layoutA == GBA_ROW_MAJOR, d.layoutB == GBA_ROW_MAJOR
    if K == 0:
        d.lda, d.ldb = (0 if row_a else M), (N if row_b else 0)
    if P is not None and K2 == 0:
        d.ldp, d.ldq = (0 if row_a else M), (N if row_b else 0)
    if bias is not None:
        if bias.dim() == 1:
            if bias.shape[0] != N or (N > 1 and bias.stride(0) != 1):
                raise ValueError("a vector bias must be a contiguous (N,) tensor")
            d.bias_kind = GBA_BIAS_ROW
        else:
            if tuple(bias.shape) != (M, N):
                raise ValueError("a matrix bias must be (M, N)")
            d.bias_kind = GBA_BIAS_FULL
            d.ldbias = _row_major_ld(bias, "bias")
        d.bias = bias.data_ptr()
        d.bias_op = OPS[bias_op]
    d.act = ACTS[act]
    d.accum = ACCS[accum]
    if out is None:
        out = torch.empty((M, N), dtype=torch.float16, device=A.device)
    if out.dim() != 2 or tuple(out.shape) != (M, N):
        raise ValueError("out must be an (M, N) matrix")
    d.C, d.ldc = out.data_ptr(), _row_major_ld(out, "out")
    d.tile_id = -1 if tile is None else int(tile)
    d.split_k = 0 if split is None else int(split)
    if isinstance(workspace, str) and workspace == "static":
        fused_gemm_desc_noalloc(d, stream, A.device)
        return out
    if workspace is not None:
        need = workspace_size(d)
        if need > 0:
            ws = stream_workspace(need, A.device, stream) if isinstance(workspace, str) else workspace
            if ws.dtype != torch.uint8 or not ws.is_cuda:
                raise TypeError("workspace must be a uint8 CUDA tensor")
            d.workspace, d.workspace_bytes = ws.data_ptr(), ws.numel()
    fused_gemm_desc(d, stream, A.device)
    return out


def bias_add_(C, bias, stream=None):
    """In place: C = fp16(C + bias[None, :]) (unfused baseline piece)."""
    M, N = C.shape
    ldc = _row_major_ld(C, "C")
    _check(lib().gba_bias_add_f16(M, N, C.data_ptr(), ldc, bias.data_ptr(),
                                  _stream_handle(stream, C.device)), "gba_bias_add_f16")
    return C


def bias_act_(C, bias, act="relu", stream=None):
    """In place: C = fp16(act(C + bias[None, :])) in one pass (the second
    kernel of the two-launch baseline)."""
    M, N = C.shape
    ldc = _row_major_ld(C, "C")
    _check(lib().gba_bias_act_f16(M, N, C.data_ptr(), ldc, bias.data_ptr(), ACTS[act],
                                  _stream_handle(stream, C.device)), "gba_bias_act_f16")
    return C


def relu_(C, stream=None):
    """In place: C = max(C, 0) (unfused baseline piece)."""
    M, N = C.shape
    ldc = _row_major_ld(C, "C")
    _check(lib().gba_relu_f16(M, N, C.data_ptr(), ldc, _stream_handle(stream, C.device)),
           "gba_relu_f16")
    return C


def add_(C, X, stream=None):
    """In place: C = fp16(C + X) (unfused baseline piece)."""
    M, N = C.shape
    if tuple(X.shape) != (M, N):
        raise ValueError("X must have the shape of C")
    _check(lib().gba_add_f16(M, N, C.data_ptr(), _row_major_ld(C, "C"), X.data_ptr(),
                             _row_major_ld(X, "X"), _stream_handle(stream, C.device)), "gba_add_f16")
    return C


def unfused_gemm_bias_relu(A, B, bias, out=None, tile=None, stream=None):
    """The three-launch baseline chain: GEMM (no epilogue), bias add, ReLU."""
    out = gemm_bias_act(A, B, None, act="none", out=out, tile=tile, stream=stream)
    bias_add_(out, bias, stream)
    relu_(out, stream)
    return out


def unfused_gemm_bias_relu_2(A, B, bias, out=None, tile=None, stream=None):
    """The two-launch baseline chain: GEMM (no epilogue), then bias add and
    ReLU in one pointwise pass."""
    out = gemm_bias_act(A, B, None, act="none", out=out, tile=tile, stream=stream)
    bias_act_(out, bias, "relu", stream)
    return out


def num_tiles():
    return lib().gba_num_tiles()


def tile_info(tile_id):
    vals = [ctypes.c_int() for _ in range(5)]
    _check(lib().gba_tile_info(int(tile_id), *[ctypes.byref(v) for v in vals]), "gba_tile_info")
    return dict(zip(("bm", "bn", "bk", "waves", "split_k"), (v.value for v in vals)))


def select_tile(M, N, K, layout_a=GBA_ROW_MAJOR, layout_b=GBA_COL_MAJOR, accum="f32", prologue=False):
    """Tile id the library would run a one-product request of this shape
    on (K: the total reduction length), -1 for the general path.  With the
    prologue the choice can differ; it is then asked through
    gba_fused_tile on a descriptor whose pointers are never dereferenced."""
    if not prologue:
        return lib().gba_select_tile(layout_a, layout_b, M, N, K, ACCS[accum])
    d = new_desc()
    d.layoutA, d.layoutB, d.M, d.N, d.K = layout_a, layout_b, M, N, K
    d.A = d.B = d.C = 1 << 16
    d.lda = K if layout_a == GBA_ROW_MAJOR else M
    d.ldb = N if layout_b == GBA_ROW_MAJOR else K
    d.ldc, d.act, d.accum, d.prologue = N, GBA_ACT_RELU, ACCS[accum], GBA_PRO_RELU
    return fused_tile(d)


def version():
    return lib().gba_version().decode()

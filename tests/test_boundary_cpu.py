"""The C ABI on the CPU: the library loads, exports every declared symbol,
and rejects bad arguments before touching the GPU.  No compute call is made
here (there is no GPU in this environment)."""
import ctypes
import os
import re

import pytest

from paper_2006_12645_amd import gba

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gba.h")

FAKE = 0x10000  # a 16-byte aligned non-null address; never dereferenced here


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(\w+)\s*\(", text, flags=re.M)))


def test_header_declares_expected_api():
    fns = declared_functions()
    assert "gemm_bias_act" in fns and "gba_bias_add_f16" in fns and "gba_relu_f16" in fns
    assert set(fns) == set(gba.SIGNATURES), (fns, sorted(gba.SIGNATURES))


def test_library_exports_every_declared_symbol():
    L = ctypes.CDLL(gba.LIB_PATH)
    for name in declared_functions():
        assert hasattr(L, name), name


def test_library_loaded_before_torch_shares_its_hip_runtime():
    """The binding loads the library after torch, whatever the caller
    imported first, so the process holds one HIP runtime (torch's) and the
    library's launches run on the runtime that owns torch's streams."""
    import json
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    code = ("import sys; sys.path.insert(0, %r)\n"
            "from paper_2006_12645_amd import gba\n"
            "gba.lib()\n"
            "import torch\n"
            "import json\n"
            "print(json.dumps(sorted({l.split()[-1] for l in open('/proc/self/maps') if 'libamdhip64' in l})))\n"
            % root)
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-2000:]
    paths = json.loads(r.stdout.strip().splitlines()[-1])
    assert len(paths) == 1, paths


def gemm(M=64, N=64, K=64, la=0, lb=1, A=FAKE, lda=None, B=FAKE, ldb=None, bias=None, C=FAKE,
         ldc=None, act=1, acc=0, tile=None):
    lda = (K if la == 0 else M) if lda is None else lda
    ldb = (N if lb == 0 else K) if ldb is None else ldb
    ldc = N if ldc is None else ldc
    args = [la, lb, M, N, K, A, lda, B, ldb, bias, C, ldc, act, acc]
    if tile is None:
        return gba.lib().gemm_bias_act(*args, None)
    return gba.lib().gemm_bias_act_tile(*args, tile, None)


@pytest.mark.parametrize("kw,status", [
    (dict(M=-1), gba.GBA_EINVAL),
    (dict(N=-5), gba.GBA_EINVAL),
    (dict(K=-1), gba.GBA_EINVAL),
    (dict(la=2), gba.GBA_EINVAL),
    (dict(lb=-1), gba.GBA_EINVAL),
    (dict(act=7), gba.GBA_EINVAL),
    (dict(acc=3), gba.GBA_EINVAL),
    (dict(ldc=63), gba.GBA_EINVAL),
    (dict(lda=63), gba.GBA_EINVAL),
    (dict(la=1, lda=63), gba.GBA_EINVAL),
    (dict(ldb=63), gba.GBA_EINVAL),
    (dict(lb=0, ldb=63), gba.GBA_EINVAL),
    (dict(A=None), gba.GBA_EINVAL),
    (dict(B=None), gba.GBA_EINVAL),
    (dict(C=None), gba.GBA_EINVAL),
    (dict(tile=gba.num_tiles()), gba.GBA_EINVAL),
    (dict(tile=1000), gba.GBA_EINVAL),
    (dict(A=FAKE + 1), gba.GBA_EUNSUPPORTED),
    (dict(C=FAKE + 1), gba.GBA_EUNSUPPORTED),
    (dict(bias=FAKE + 1), gba.GBA_EUNSUPPORTED),
    (dict(M=2**31), gba.GBA_EUNSUPPORTED),
    (dict(K=2**31, lda=2**31), gba.GBA_EUNSUPPORTED),
    # empty output: accepted, nothing launched (NULL operands are fine)
    (dict(M=0, A=None, B=None, C=None), gba.GBA_OK),
    (dict(N=0, A=None, B=None, C=None), gba.GBA_OK),
    (dict(M=0, tile=3), gba.GBA_OK),
])
def test_gemm_validation(kw, status):
    assert gemm(**kw) == status


def test_pointwise_validation():
    L = gba.lib()
    assert L.gba_bias_add_f16(-1, 4, FAKE, 4, FAKE, None) == gba.GBA_EINVAL
    assert L.gba_bias_add_f16(4, 4, None, 4, FAKE, None) == gba.GBA_EINVAL
    assert L.gba_bias_add_f16(4, 4, FAKE, 4, None, None) == gba.GBA_EINVAL
    assert L.gba_bias_add_f16(4, 8, FAKE, 4, FAKE, None) == gba.GBA_EINVAL
    assert L.gba_bias_add_f16(4, 4, FAKE + 1, 4, FAKE, None) == gba.GBA_EUNSUPPORTED
    assert L.gba_bias_add_f16(0, 4, None, 4, None, None) == gba.GBA_OK
    assert L.gba_relu_f16(4, -4, FAKE, 4, None) == gba.GBA_EINVAL
    assert L.gba_relu_f16(4, 4, None, 4, None) == gba.GBA_EINVAL
    assert L.gba_relu_f16(2**31, 4, FAKE, 4, None) == gba.GBA_EUNSUPPORTED
    assert L.gba_relu_f16(4, 0, None, 0, None) == gba.GBA_OK
    assert L.gba_bias_act_f16(-1, 4, FAKE, 4, FAKE, 1, None) == gba.GBA_EINVAL
    assert L.gba_bias_act_f16(4, 4, FAKE, 4, None, 1, None) == gba.GBA_EINVAL
    assert L.gba_bias_act_f16(4, 4, FAKE, 4, FAKE, 9, None) == gba.GBA_EINVAL
    assert L.gba_bias_act_f16(4, 4, FAKE + 1, 4, FAKE, 1, None) == gba.GBA_EUNSUPPORTED
    assert L.gba_bias_act_f16(0, 4, None, 4, None, 1, None) == gba.GBA_OK


def test_tile_table():
    n = gba.num_tiles()
    assert n >= 1
    for t in range(n):
        info = gba.tile_info(t)
        assert info["bm"] % 16 == 0 and info["bn"] % 32 == 0 and info["bk"] % 32 == 0
        assert 1 <= info["waves"] <= 16 and info["split_k"] in (1, 2, 4)
        # two LDS stages of split_k x (bm + bn) x bk fp16 fit in a gfx950 CU's 160 KB
        assert 2 * info["split_k"] * (info["bm"] + info["bn"]) * info["bk"] * 2 <= 160 * 1024
    with pytest.raises(gba.GbaError):
        gba.tile_info(n)


@pytest.mark.parametrize("shape", [(128, 128, 128), (1024, 1024, 1024), (4096, 4096, 4096),
                                   (8192, 4096, 1024), (8192, 1024, 4096), (32, 4096, 1024),
                                   (128, 4096, 1024), (256, 4096, 1024), (1000, 1000, 1000),
                                   (1, 1, 1), (0, 5, 5)])
def test_select_tile(shape):
    t = gba.select_tile(*shape)
    M, N, _ = shape
    if M < 32 or N < 32:
        assert t == -1
    else:
        assert 0 <= t < gba.num_tiles()
        info = gba.tile_info(t)
        assert info["bm"] <= M and info["bn"] <= N


def test_select_tile_split_k_policy():
    # long reduction, few output tiles: split-K with fp32 accumulation only
    t = gba.select_tile(64, 512, 32768)
    assert gba.tile_info(t)["split_k"] > 1
    t16 = gba.select_tile(64, 512, 32768, accum="f16")
    assert gba.tile_info(t16)["split_k"] == 1
    # enough output tiles: no split-K
    assert gba.tile_info(gba.select_tile(4096, 4096, 8192))["split_k"] == 1


def test_select_tile_rejects_bad_input():
    assert gba.lib().gba_select_tile(0, 1, -1, 4, 4, 0) == -1
    assert gba.lib().gba_select_tile(5, 1, 1, 4, 4, 0) == -1
    assert gba.lib().gba_select_tile(0, 1, 1, 4, 4, 9) == -1


def test_status_strings_and_version():
    for s in range(5):
        assert gba.lib().gba_status_string(s)
    assert b"unknown" in gba.lib().gba_status_string(99)
    assert "gfx950" in gba.version()


def test_layout_inference_on_cpu_tensors():
    import torch
    a = torch.zeros(6, 10, dtype=torch.float16)
    assert gba.operand_layout(a, 6, 10) == (gba.GBA_ROW_MAJOR, 10)
    assert gba.operand_layout(a.t(), 10, 6) == (gba.GBA_COL_MAJOR, 10)
    assert gba.operand_layout(a[:, :7], 6, 7) == (gba.GBA_ROW_MAJOR, 10)
    with pytest.raises(ValueError):
        gba.operand_layout(a[::2, ::2], 3, 5)


def test_fused_desc_matches_c_layout(tmp_path):
    """The ctypes mirror of struct gba_fused_desc has the C compiler's
    size and field offsets."""
    import subprocess
    fields = [f[0] for f in gba.FusedDesc._fields_]
    prog = tmp_path / "desc.c"
    prog.write_text("#include <stdio.h>\n#include <stddef.h>\n#include \"gba.h\"\nint main(void){\n"
                    "printf(\"%zu\\n\", sizeof(gba_fused_desc));\n" +
                    "".join(f"printf(\"%zu\\n\", offsetof(gba_fused_desc, {f}));\n" for f in fields) +
                    "return 0;}\n")
    exe = tmp_path / "desc"
    subprocess.run(["gcc", "-std=c99", "-I", os.path.join(ROOT, "include"), "-o", str(exe), str(prog)],
                   check=True)
    vals = [int(x) for x in subprocess.run([str(exe)], capture_output=True, text=True,
                                           check=True).stdout.split()]
    assert vals[0] == ctypes.sizeof(gba.FusedDesc)
    assert vals[1:] == [getattr(gba.FusedDesc, f).offset for f in fields]


def test_fused_desc_defaults():
    d = gba.new_desc()
    assert (d.layoutA, d.layoutB, d.prologue, d.second, d.bias_kind, d.bias_op, d.act,
            d.accum, d.tile_id, d.split_k) == (0, 0, 0, 0, 0, 0, 0, 0, -1, 0)
    assert d.A is None and d.C is None and d.M == 0 and d.K2 == 0
    assert d.workspace is None and d.workspace_bytes == 0
    gba.lib().gba_fused_desc_init(None)  # ignored, no crash


def fused(**kw):
    """gba_fused_gemm on a valid 64^3 request with two products, a full
    bias and ReLU, modified by kw (pointers are never dereferenced: every
    case is rejected or empty before any launch)."""
    d = gba.new_desc()
    d.layoutA, d.layoutB, d.M, d.N, d.K = 0, 1, 64, 64, 64
    d.A, d.lda, d.B, d.ldb = FAKE, 64, FAKE, 64
    d.second, d.K2, d.P, d.ldp, d.Q, d.ldq = gba.GBA_SECOND_ADD, 32, FAKE, 32, FAKE, 32
    d.bias_kind, d.bias, d.ldbias = gba.GBA_BIAS_FULL, FAKE, 64
    d.act, d.C, d.ldc = gba.GBA_ACT_RELU, FAKE, 64
    for k, v in kw.items():
        setattr(d, k, v)
    return gba.lib().gba_fused_gemm(ctypes.byref(d), None)


@pytest.mark.parametrize("kw,status", [
    (dict(prologue=2), gba.GBA_EINVAL),
    (dict(second=3), gba.GBA_EINVAL),
    (dict(second=-1), gba.GBA_EINVAL),
    (dict(bias_kind=3), gba.GBA_EINVAL),
    (dict(bias_op=2), gba.GBA_EINVAL),
    (dict(act=4), gba.GBA_EINVAL),
    (dict(act=-1), gba.GBA_EINVAL),
    (dict(accum=2), gba.GBA_EINVAL),
    (dict(tile_id=gba.num_tiles()), gba.GBA_EINVAL),
    (dict(K2=-1), gba.GBA_EINVAL),
    (dict(ldp=31), gba.GBA_EINVAL),
    (dict(layoutA=1, ldp=63), gba.GBA_EINVAL),
    (dict(ldq=31), gba.GBA_EINVAL),
    (dict(layoutB=0, ldq=63), gba.GBA_EINVAL),
    (dict(P=None), gba.GBA_EINVAL),
    (dict(Q=None), gba.GBA_EINVAL),
    (dict(bias=None), gba.GBA_EINVAL),
    (dict(ldbias=63), gba.GBA_EINVAL),
    (dict(ldbias=-1), gba.GBA_EINVAL),
    (dict(C=None), gba.GBA_EINVAL),
    (dict(A=None), gba.GBA_EINVAL),
    (dict(P=FAKE + 1), gba.GBA_EUNSUPPORTED),
    (dict(Q=FAKE + 1), gba.GBA_EUNSUPPORTED),
    (dict(K2=2**31, ldp=2**31), gba.GBA_EUNSUPPORTED),
    # with no second product, P/Q/K2 are not read; a row bias ignores ldbias
    (dict(second=0, P=None, Q=None, K2=-7, ldp=-1, M=0), gba.GBA_OK),
    (dict(bias_kind=gba.GBA_BIAS_ROW, ldbias=-3, N=0), gba.GBA_OK),
    (dict(M=0, A=None, B=None, P=None, Q=None, C=None, bias=None), gba.GBA_OK),
    (dict(split_k=-1), gba.GBA_EINVAL),
    (dict(workspace=FAKE + 16, workspace_bytes=1 << 20), gba.GBA_EINVAL),
    (dict(split_k=-1, M=0), gba.GBA_EINVAL),
])
def test_fused_validation(kw, status):
    assert fused(**kw) == status


def test_fused_validation_null_desc():
    assert gba.lib().gba_fused_gemm(None, None) == gba.GBA_EINVAL


def ws_bytes(**kw):
    """gba_fused_workspace_size of an aligned one-product RC request
    (M = N = 512, K = 320: five 64-deep steps), modified by kw."""
    d = gba.new_desc()
    d.layoutA, d.layoutB, d.M, d.N, d.K = 0, 1, 512, 512, 320
    d.A, d.lda, d.B, d.ldb, d.C, d.ldc = FAKE, 320, FAKE, 320, FAKE, 512
    for k, v in kw.items():
        setattr(d, k, v)
    n = ctypes.c_size_t(12345)
    st = gba.lib().gba_fused_workspace_size(ctypes.byref(d), ctypes.byref(n))
    return st, n.value


def expected_ws(tile, M, N, splits):
    info = gba.tile_info(tile)
    tiles = -(-M // info["bm"]) * -(-N // info["bn"])
    return -(-tiles * 4 // 256) * 256 + splits * tiles * info["bm"] * info["bn"] * 4


@pytest.mark.parametrize("tile,split_k,splits", [
    (4, 2, 2),    # 5 steps: ranges of 3 and 2
    (4, 3, 3),    # ranges of 2, 2, 1
    (4, 4, 3),    # ranges of 2 cover the 5 steps in 3 splits
    (4, 5, 5),
    (4, 9, 5),    # no more splits than steps
    (6, 2, 2),
    (9, 5, 5),
])
def test_workspace_size_of_forced_splits(tile, split_k, splits):
    assert ws_bytes(tile_id=tile, split_k=split_k) == (gba.GBA_OK, expected_ws(tile, 512, 512, splits))


@pytest.mark.parametrize("kw", [
    dict(tile_id=4, split_k=1),                  # never split
    dict(tile_id=10, split_k=4),                 # a tile with k-groups inside the workgroup
    dict(tile_id=1, split_k=4),                  # 256x256: no split variant
    dict(tile_id=4, split_k=4, accum=gba.GBA_ACC_F16),
    dict(tile_id=4, split_k=4, A=FAKE + 2),      # general path
    dict(tile_id=4, split_k=4, K=0),             # no reduction steps
    dict(tile_id=4, split_k=4, K=64),            # one step
    dict(tile_id=4, split_k=4, M=0),             # empty output
])
def test_workspace_size_without_split(kw):
    assert ws_bytes(**kw) == (gba.GBA_OK, 0)


@pytest.mark.parametrize("M,N,K,splits", [
    (64, 512, 32768, 16),      # 8 tiles of 64x64: 128 workgroups
    (128, 128, 65536, 32),     # 4 tiles
    (64, 2048, 16384, 4),      # 32 tiles
    (64, 2048, 16320, 0),      # reduction below 16384: no split
    (512, 512, 32768, 0),      # 64 tiles: enough workgroups unsplit
    (32, 512, 32768, 0),       # smaller than the 64x64 tile
])
def test_workspace_size_of_the_library_split(M, N, K, splits):
    st, n = ws_bytes(M=M, N=N, K=K, lda=K, ldb=K, ldc=N)
    assert (st, n) == (gba.GBA_OK, expected_ws(6, M, N, splits) if splits else 0)
    # never for fp16 accumulation or a requested tile
    assert ws_bytes(M=M, N=N, K=K, lda=K, ldb=K, ldc=N, accum=gba.GBA_ACC_F16) == (gba.GBA_OK, 0)
    assert ws_bytes(M=M, N=N, K=K, lda=K, ldb=K, ldc=N, tile_id=8) == (gba.GBA_OK, 0)


def test_workspace_size_counts_both_products():
    # 5 + 3 steps of A.B and P.Q split 4 ways: ranges of 2
    st, n = ws_bytes(tile_id=4, split_k=4, second=gba.GBA_SECOND_SUB, K2=192, P=FAKE, ldp=192,
                     Q=FAKE, ldq=192)
    assert (st, n) == (gba.GBA_OK, expected_ws(4, 512, 512, 4))


def test_workspace_size_errors():
    assert ws_bytes(split_k=-2)[0] == gba.GBA_EINVAL
    assert ws_bytes(act=9)[0] == gba.GBA_EINVAL
    d = gba.new_desc()
    assert gba.lib().gba_fused_workspace_size(ctypes.byref(d), None) == gba.GBA_EINVAL
    n = ctypes.c_size_t(0)
    assert gba.lib().gba_fused_workspace_size(None, ctypes.byref(n)) == gba.GBA_EINVAL


def test_generalised_act_enum_accepted_by_gemm_bias_act():
    # sigmoid and tanh pass validation (an empty problem launches nothing)
    assert gemm(M=0, act=gba.GBA_ACT_SIGMOID) == gba.GBA_OK
    assert gemm(M=0, act=gba.GBA_ACT_TANH) == gba.GBA_OK
    assert gemm(act=4) == gba.GBA_EINVAL


def test_operand_layout_with_required_layout():
    import torch
    p = torch.zeros(1, 9, dtype=torch.float16)
    assert gba.operand_layout(p, 1, 9, want=gba.GBA_COL_MAJOR) == (gba.GBA_COL_MAJOR, 1)
    assert gba.operand_layout(p, 1, 9, want=gba.GBA_ROW_MAJOR) == (gba.GBA_ROW_MAJOR, 9)
    q = torch.zeros(6, 10, dtype=torch.float16)
    with pytest.raises(ValueError):
        gba.operand_layout(q, 6, 10, want=gba.GBA_COL_MAJOR)


def test_add_validation():
    L = gba.lib()
    assert L.gba_add_f16(-1, 4, FAKE, 4, FAKE, 4, None) == gba.GBA_EINVAL
    assert L.gba_add_f16(4, 4, FAKE, 4, None, 4, None) == gba.GBA_EINVAL
    assert L.gba_add_f16(4, 4, FAKE, 4, FAKE, 3, None) == gba.GBA_EINVAL
    assert L.gba_add_f16(4, 4, FAKE, 4, FAKE + 1, 4, None) == gba.GBA_EUNSUPPORTED
    assert L.gba_add_f16(0, 4, None, 4, None, 4, None) == gba.GBA_OK


class _FakeStream:
    cuda_stream = 0x1234


def test_auto_workspace_refused_during_capture(monkeypatch):
    """workspace='auto' must not allocate or zero-fill a buffer while the
    stream is being captured into a graph (that work would be captured)."""
    from paper_2006_12645_amd import gba
    monkeypatch.setattr(gba, "_workspaces", {})
    monkeypatch.setattr(gba, "stream_capturing", lambda s: True)
    with pytest.raises(RuntimeError, match="captured"):
        gba.stream_workspace(1 << 20, "cuda:0", _FakeStream())


def test_auto_workspace_reused_during_capture(monkeypatch):
    """A workspace cached by an earlier eager call is handed out during
    capture without any new allocation, and a replaced one is kept alive."""
    from paper_2006_12645_amd import gba
    cached = type("T", (), {"numel": lambda self: 4 << 20})()
    monkeypatch.setattr(gba, "_workspaces", {(0, _FakeStream.cuda_stream): cached})
    monkeypatch.setattr(gba, "stream_capturing", lambda s: True)
    assert gba.stream_workspace(1 << 20, "cuda:0", _FakeStream()) is cached
    with pytest.raises(RuntimeError):
        gba.stream_workspace(8 << 20, "cuda:0", _FakeStream())


def test_noalloc_rejects_a_split_beyond_its_scratch():
    """gba_fused_gemm_noalloc refuses, before any launch, a split whose
    workspace exceeds the library's static scratch; it validates like
    gba_fused_gemm."""
    L = gba.lib()
    d = gba.new_desc()
    d.layoutA, d.layoutB = gba.GBA_ROW_MAJOR, gba.GBA_COL_MAJOR
    d.M, d.N, d.K = 1024, 1024, 8192
    d.A = d.B = d.C = FAKE
    d.lda, d.ldb, d.ldc = 8192, 8192, 1024
    d.tile_id, d.split_k = 4, 64          # 64 tiles of 128x128, 64 splits each
    assert gba.workspace_size(d) > gba.GBA_NOALLOC_SCRATCH_BYTES
    assert L.gba_fused_gemm_noalloc(ctypes.byref(d), None) == gba.GBA_ESCRATCH
    assert b"scratch" in L.gba_status_string(gba.GBA_ESCRATCH)
    d.M = -1
    assert L.gba_fused_gemm_noalloc(ctypes.byref(d), None) == gba.GBA_EINVAL
    assert L.gba_fused_gemm_noalloc(None, None) == gba.GBA_EINVAL


def test_shared_layout_of_a_and_p():
    """A and P (and B and Q) are passed in one layout; an operand with a
    single row or column fits either, so the other one decides, and two
    operands stored in different layouts are refused."""
    torch = pytest.importorskip("torch")
    row = lambda r, c, ld: torch.empty(r, ld, dtype=torch.float16)[:, :c]
    col = lambda r, c, ld: torch.empty(c, ld, dtype=torch.float16)[:, :r].t()
    R, C = gba.GBA_ROW_MAJOR, gba.GBA_COL_MAJOR
    # K = 1: A (48 x 1) is a single column, P decides
    assert gba.shared_layout(col(48, 1, 56), 48, 1, col(48, 456, 56), 48, 456) == C
    assert gba.shared_layout(col(48, 1, 56), 48, 1, row(48, 456, 464), 48, 456) == R
    assert gba.operand_layout(col(48, 1, 56), 48, 1, want=C) == (C, 48)
    # B (1 x 312) is a single row, Q decides
    assert gba.shared_layout(row(1, 312, 320), 1, 312, col(456, 312, 464), 456, 312) == C
    assert gba.shared_layout(row(64, 32, 40), 64, 32, row(64, 16, 24), 64, 16) == R
    with pytest.raises(ValueError):
        gba.shared_layout(row(64, 32, 40), 64, 32, col(64, 16, 72), 64, 16)

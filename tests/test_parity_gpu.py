"""HIP path vs the CPU oracle, element by element, through the C ABI.

Each case prints its name, shape and seed before touching the GPU so a
failing run names the case.  Inputs come from the seeded generators in
paper_2006_12645_amd.datagen; expected values from the oracle only.
"""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2006_12645_amd import datagen as D
from paper_2006_12645_amd import gba

import gpu_util as U

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

LAYOUTS = ["RR", "RC", "CR", "CC"]
NUM_TILES = 26
SPLITK_TILES = [10, 11, 12, 13, 14, 15]


def announce(*what):
    print("CASE", *what, flush=True)


def run_gpu(A, B, bias, layout, act="relu", accum="f32", tile=None, pad=0, out=None, stream=None):
    la, lb = D.LAYOUT_NAMES[layout]
    dA = U.device_operand(A, la, pad)
    dB = U.device_operand(B, lb, pad)
    dbias = None if bias is None else torch.from_numpy(bias).cuda()
    o = gba.gemm_bias_act(dA, dB, dbias, act=act, accum=accum, tile=tile, out=out, stream=stream)
    torch.cuda.synchronize()
    return o


@pytest.fixture(autouse=True, scope="module")
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    gba.lib()
    yield


# ----------------------------------------------------------------------------
# The five workload families

def test_cube128_rc():
    w = D.WORKLOADS["cube128_RC"]
    announce(w.name)
    A, B, bias = D.logical_inputs(w)
    got = run_gpu(A, B, bias, "RC").cpu().numpy()
    U.assert_close(got, U.oracle_for(A, B, bias), what=w.name)


@pytest.fixture(scope="module")
def cube1024():
    w = D.WORKLOADS["cube1024_all_layouts"]
    A, B, bias = D.logical_inputs(w)
    return A, B, bias, U.oracle_for(A, B, bias)


@pytest.mark.parametrize("layout", LAYOUTS)
def test_cube1024_layouts(cube1024, layout):
    A, B, bias, ref = cube1024
    announce("cube1024", layout)
    U.assert_close(run_gpu(A, B, bias, layout).cpu().numpy(), ref, what=f"1024^3 {layout}")


@pytest.fixture(scope="module")
def cube4096():
    """The 4096^3 headline inputs and the oracle over EVERY output: the fused
    result (bias + ReLU) and the plain product (no bias, no activation)."""
    w = D.WORKLOADS["cube4096_RC"]
    A, B, bias = D.logical_inputs(w)
    ref_fused = U.oracle_for(A, B, bias)
    ref_plain = U.oracle_for(A, B, None, act=O.ACT_NONE)
    return A, B, bias, ref_fused, ref_plain


def test_cube4096_fused_full(cube4096):
    A, B, bias, ref, _ = cube4096
    announce("cube4096 fused RC, every output")
    got = run_gpu(A, B, bias, "RC").cpu().numpy()
    U.assert_close(got, ref, what="4096^3 fused")


def test_cube4096_plain_full(cube4096):
    A, B, _, _, ref = cube4096
    announce("cube4096 plain RC, every output")
    got = run_gpu(A, B, None, "RC", act="none").cpu().numpy()
    U.assert_close(got, ref, what="4096^3 plain")


def test_cube4096_unfused_full(cube4096):
    A, B, bias, ref, _ = cube4096
    announce("cube4096 unfused RC, every output")
    dA = U.device_operand(A, D.ROW)
    dB = U.device_operand(B, D.COL)
    out = gba.unfused_gemm_bias_relu(dA, dB, torch.from_numpy(bias).cuda())
    torch.cuda.synchronize()
    U.assert_close(out.cpu().numpy(), ref, what="unfused")


@pytest.mark.parametrize("name", ["mlp_up_8192x4096x1024", "mlp_down_8192x1024x4096"])
def test_mlp_full(name):
    w = D.WORKLOADS[name]
    announce(name, "every output")
    A, B, bias = D.logical_inputs(w)
    got = run_gpu(A, B, bias, "RC").cpu().numpy()
    U.assert_close(got, U.oracle_for(A, B, bias), what=name)


@pytest.mark.parametrize("name", ["infer_m32_n4096_k1024", "infer_m128_n4096_k1024",
                                  "infer_m256_n4096_k1024"])
@pytest.mark.parametrize("accum", ["f32", "f16"])
def test_inference_shapes(name, accum):
    w = D.WORKLOADS[name]
    announce(name, accum)
    A, B, bias = D.logical_inputs(w)
    got = run_gpu(A, B, bias, "RC", accum=accum).cpu().numpy()
    U.assert_close(got, U.oracle_for(A, B, bias), accum=accum, what=f"{name} {accum}")


@pytest.fixture(scope="module")
def ragged():
    w = D.WORKLOADS["ragged1000"]
    A, B, bias = D.logical_inputs(w)
    return A, B, bias, U.oracle_for(A, B, bias)


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("accum", ["f32", "f16"])
def test_ragged1000(ragged, layout, accum):
    A, B, bias, ref = ragged
    announce("ragged1000", layout, accum)
    got = run_gpu(A, B, bias, layout, accum=accum).cpu().numpy()
    U.assert_close(got, ref, accum=accum, what=f"1000^3 {layout} {accum}")


# ----------------------------------------------------------------------------
# Exactness, tiles, edges

@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("accum", ["f32", "f16"])
def test_integer_data_bit_exact(layout, accum):
    """{-1,0,1} operands and integer bias: every partial sum is an integer
    below 2048, exact in fp16 and fp32, so the result must equal the oracle
    exactly whatever the summation order or accumulator precision."""
    M, N, K = 300, 260, 1000
    announce("integer exact", layout, accum, M, N, K)
    A, B, bias = D.random_problem(77, M, N, K, dist="int")
    got = run_gpu(A, B, bias, layout, accum=accum).cpu().numpy().astype(np.float64)
    assert np.array_equal(got, U.oracle_for(A, B, bias))


def test_tile_count():
    assert gba.num_tiles() == NUM_TILES


@pytest.mark.parametrize("tile", range(NUM_TILES))
@pytest.mark.parametrize("layout", LAYOUTS)
def test_every_tile_config(tile, layout):
    """Fast path (sizes multiples of 8, ragged against every tile)."""
    M, N, K = 296, 328, 200
    announce("tile", tile, layout)
    A, B, bias = D.random_problem(1000 + tile, M, N, K)
    got = run_gpu(A, B, bias, layout, tile=tile).cpu().numpy()
    U.assert_close(got, U.oracle_for(A, B, bias), what=f"tile {tile} {layout}")


@pytest.mark.parametrize("tile", [11, 13])
@pytest.mark.parametrize("K", [64, 200, 1000, 5000])
def test_deep_pipeline_short_and_long_k(tile, K):
    """Four-stage pipelines with fewer reduction steps than stages (the
    trailing copies re-fetch the last step) and with many steps."""
    M, N = 136, 200
    announce("deep", tile, K)
    A, B, bias = D.random_problem(3000 + tile + K, M, N, K)
    got = run_gpu(A, B, bias, "RC", tile=tile).cpu().numpy()
    U.assert_close(got, U.oracle_for(A, B, bias), what=f"deep tile {tile} K={K}")


@pytest.mark.parametrize("tile", [None, 1, 4, 6, 9, 11, 13])
@pytest.mark.parametrize("K", [1, 5, 77, 130])
def test_mn_contiguous_operands_any_k(tile, K):
    """Column-major A with row-major B keeps the fast path for any K (both
    operands are contiguous along M / N): reduction rows past K in the last
    step are zero-filled row by row."""
    M, N = 264, 296
    announce("CR any K", tile, K)
    A, B, bias = D.random_problem(3500 + K, M, N, K)
    got = run_gpu(A, B, bias, "CR", tile=tile).cpu().numpy()
    U.assert_close(got, U.oracle_for(A, B, bias), what=f"CR tile {tile} K={K}")


@pytest.mark.parametrize("layout", ["RR", "CR", "CC"])
@pytest.mark.parametrize("tile", [11, 13])
def test_deep_pipeline_transposed_layouts(layout, tile):
    M, N, K = 136, 200, 5000
    announce("deep", layout, tile)
    A, B, bias = D.random_problem(3600 + tile, M, N, K)
    got = run_gpu(A, B, bias, layout, tile=tile).cpu().numpy()
    U.assert_close(got, U.oracle_for(A, B, bias), what=f"deep {layout} tile {tile}")


def test_long_k_selects_split_k():
    """A long reduction over few output tiles takes the split-K tile."""
    M, N, K = 96, 320, 8192
    announce("long-K selection")
    assert gba.tile_info(gba.select_tile(M, N, K))["split_k"] > 1
    A, B, bias = D.random_problem(3100, M, N, K)
    got = run_gpu(A, B, bias, "RC").cpu().numpy()
    U.assert_close(got, U.oracle_for(A, B, bias), what="long-K")


@pytest.mark.parametrize("tile", range(NUM_TILES))
def test_every_tile_config_f16acc(tile):
    M, N, K = 136, 248, 520
    announce("tile f16acc", tile)
    A, B, bias = D.random_problem(1100 + tile, M, N, K)
    got = run_gpu(A, B, bias, "RC", accum="f16", tile=tile).cpu().numpy()
    U.assert_close(got, U.oracle_for(A, B, bias), accum="f16", what=f"tile {tile} f16")


@pytest.mark.parametrize("tile", SPLITK_TILES)
@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("K", [64, 104, 136, 1000])
def test_split_k_partial_slabs(tile, layout, K):
    """Intra-workgroup split-K with reduction lengths that leave some k-groups
    a partial slab or none at all in the last step."""
    M, N = 136, 200
    announce("split-K", tile, layout, K)
    A, B, bias = D.random_problem(2000 + tile * 7 + K, M, N, K)
    got = run_gpu(A, B, bias, layout, tile=tile).cpu().numpy()
    U.assert_close(got, U.oracle_for(A, B, bias), what=f"split-K tile {tile} {layout} K={K}")


def test_split_k_integer_bit_exact():
    """Split-K sums partials in a different order; on integer data the result
    is still exact."""
    M, N, K = 192, 256, 2040
    announce("split-K integer exact")
    A, B, bias = D.random_problem(78, M, N, K, dist="int")
    for tile in SPLITK_TILES:
        got = run_gpu(A, B, bias, "RC", tile=tile).cpu().numpy().astype(np.float64)
        assert np.array_equal(got, U.oracle_for(A, B, bias)), tile


RAGGED = [1, 7, 31, 33, 127, 129]


@pytest.mark.parametrize("M", RAGGED)
@pytest.mark.parametrize("N", [1, 33, 129])
@pytest.mark.parametrize("K", [7, 33, 129])
def test_ragged_sizes_guarded(M, N, K):
    """Odd sizes in every dimension (scalar path when a leading dimension is
    not a multiple of 8), with a sentinel-filled guard band around C that
    must come back untouched."""
    announce("ragged", M, N, K)
    A, B, bias = D.random_problem(M * 10000 + N * 100 + K, M, N, K)
    pad = (-K) % 8 if K % 8 else 0
    G = 8
    big = torch.full((M + 2 * G, N + 2 * G), 12345.0, dtype=torch.float16, device="cuda")
    out = big[G:G + M, G:G + N]
    for layout in LAYOUTS:
        big.fill_(12345.0)
        run_gpu(A, B, bias, layout, out=out, pad=pad)
        host = big.cpu().numpy()
        inner = host[G:G + M, G:G + N]
        U.assert_close(inner, U.oracle_for(A, B, bias), what=f"{M}x{N}x{K} {layout}")
        guard = host.copy()
        guard[G:G + M, G:G + N] = 12345.0
        assert (guard == np.float16(12345.0)).all(), "write outside C"


def test_unaligned_operands_take_scalar_path():
    M, N, K = 200, 150, 300
    announce("unaligned")
    A, B, bias = D.random_problem(55, M, N, K)
    ref = U.oracle_for(A, B, bias)
    for layout in LAYOUTS:
        la, lb = D.LAYOUT_NAMES[layout]
        # operands shifted by one fp16 element inside a larger buffer
        sa = D.store(A, la, (K if la == D.ROW else M) + 3)
        sb = D.store(B, lb, (N if lb == D.ROW else K) + 3)
        # storage that starts one fp16 element past a 16-byte boundary
        ta = torch.empty(1 + sa.size, dtype=torch.float16, device="cuda")
        tb = torch.empty(1 + sb.size, dtype=torch.float16, device="cuda")
        ta[1:] = torch.from_numpy(sa.ravel()).cuda()
        tb[1:] = torch.from_numpy(sb.ravel()).cuda()
        ta, tb = ta[1:], tb[1:]
        lda, ldb = sa.shape[1], sb.shape[1]
        dA = (ta.as_strided((M, K), (lda, 1)) if la == D.ROW else ta.as_strided((M, K), (1, lda)))
        dB = (tb.as_strided((K, N), (ldb, 1)) if lb == D.ROW else tb.as_strided((K, N), (1, ldb)))
        got = gba.gemm_bias_act(dA, dB, torch.from_numpy(bias).cuda(), act="relu")
        torch.cuda.synchronize()
        U.assert_close(got.cpu().numpy(), ref, what=f"unaligned {layout}")


def test_k_zero_gives_activation_of_bias():
    M, N = 70, 90
    announce("K=0")
    bias = D.uniform_f16(5, (N,))
    A = torch.zeros((M, 0), dtype=torch.float16, device="cuda")
    B = torch.zeros((0, N), dtype=torch.float16, device="cuda")
    for act in ("relu", "none"):
        got = gba.gemm_bias_act(A, B, torch.from_numpy(bias).cuda(), act=act)
        torch.cuda.synchronize()
        want = np.maximum(bias.astype(np.float64), 0) if act == "relu" else bias.astype(np.float64)
        assert np.array_equal(got.cpu().numpy().astype(np.float64), np.broadcast_to(want, (M, N)))


def test_no_bias_no_activation_matches_oracle():
    M, N, K = 257, 511, 384
    announce("plain")
    A, B, _ = D.random_problem(66, M, N, K)
    for layout in LAYOUTS:
        got = run_gpu(A, B, None, layout, act="none").cpu().numpy()
        U.assert_close(got, U.oracle_for(A, B, None, act=O.ACT_NONE), what=f"plain {layout}")


def test_relu_output_properties():
    M, N, K = 512, 512, 512
    announce("relu props")
    A, B, bias = D.random_problem(67, M, N, K)
    got = run_gpu(A, B, bias, "RC").cpu().numpy().astype(np.float64)
    pre = U.oracle_for(A, B, bias, act=O.ACT_NONE)
    assert (got >= 0).all()
    assert (got[pre < -0.02] == 0).all()
    assert ((got > 0) == (pre > 0))[np.abs(pre) > 0.02].all()


def test_deterministic_and_stream():
    M, N, K = 1024, 768, 512
    announce("determinism")
    A, B, bias = D.random_problem(68, M, N, K)
    a = run_gpu(A, B, bias, "RC")
    b = run_gpu(A, B, bias, "RC")
    assert torch.equal(a, b)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        c = run_gpu(A, B, bias, "RC", stream=s)
    s.synchronize()
    assert torch.equal(a, c)


def test_graph_capture_replays():
    """The fused kernels captured in a HIP graph (a plain call, a call with
    the reduction split across workgroups through a caller workspace, the
    transposed layout, and two small tiles whose copies run on waves of
    their own, one with fp16 accumulation) replay to the eager results,
    replay after replay, with eager work of the library on the same buffers
    in between."""
    announce("graph capture")
    M, N, K = 384, 256, 4096
    A, B, bias = D.random_problem(69, M, N, K)
    dA, dB = U.device_operand(A, D.ROW), U.device_operand(B, D.COL)
    dAc, dBr = U.device_operand(A, D.COL), U.device_operand(B, D.ROW)
    dbias = torch.from_numpy(bias).cuda()
    ws = torch.zeros(16 << 20, dtype=torch.uint8, device="cuda")
    outs = [torch.empty(M, N, dtype=torch.float16, device="cuda") for _ in range(5)]
    calls = [lambda: gba.gemm_bias_act(dA, dB, dbias, out=outs[0]),
             lambda: gba.fused_gemm(dA, dB, bias=dbias, tile=6, split=8, workspace=ws, out=outs[1]),
             lambda: gba.fused_gemm(dAc, dBr, bias=dbias, act="tanh", out=outs[2]),
             lambda: gba.fused_gemm(dA, dBr, bias=dbias, tile=24, out=outs[3]),
             lambda: gba.fused_gemm(dA, dB, bias=dbias, tile=21, accum="f16", out=outs[4])]
    for f in calls:
        f()
    torch.cuda.synchronize()
    eager = [o.clone() for o in outs]
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        for f in calls:
            f()
    torch.cuda.synchronize()
    for rep in range(4):
        for o in outs:
            o.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        for o, e in zip(outs, eager):
            assert torch.equal(o, e), f"replay {rep}"
        # eager work in between, on the same workspace and outputs
        calls[1]()
        calls[0]()
        torch.cuda.synchronize()
    assert not ws[:(M // 64) * (N // 64) * 4].any().item()  # the split's counters are back at 0


def test_cube4096_two_launch_chain_full(cube4096):
    """The two-launch baseline (GEMM, then bias add and ReLU in one pass),
    every output against the oracle."""
    A, B, bias, ref, _ = cube4096
    announce("cube4096 two-launch chain RC, every output")
    out = gba.unfused_gemm_bias_relu_2(U.device_operand(A, D.ROW), U.device_operand(B, D.COL),
                                       torch.from_numpy(bias).cuda())
    torch.cuda.synchronize()
    U.assert_close(out.cpu().numpy(), ref, what="two-launch chain")


@pytest.mark.parametrize("act", ["none", "relu", "sigmoid", "tanh"])
def test_bias_act_piece(act):
    """gba_bias_act_f16 against the oracle's activations: the input C stands
    for a matmul result, so the oracle evaluates act(I.C + bias) with an
    identity left operand (exact), and the kernel's one fp16 rounding of the
    fp32 result must be within the fp32-accumulation bound; the aligned and
    the scalar (odd leading dimension) paths."""
    M, N = 64, 1031
    announce("bias_act", act)
    C0 = D.uniform_f16(92, (M, N), -4, 4)
    bias = D.uniform_f16(93, (N,))
    eye = np.eye(M, dtype=np.float16)
    ref = O.fused(D.store(eye, D.ROW), D.ROW, D.store(C0, D.ROW), D.ROW, M, N, M, bias=bias,
                  act={"none": O.ACT_NONE, "relu": O.ACT_RELU, "sigmoid": O.ACT_SIGMOID,
                       "tanh": O.ACT_TANH}[act])
    for pad in (0, 1):
        C = U.device_operand(C0, D.ROW, pad=pad)
        gba.bias_act_(C, torch.from_numpy(bias).cuda(), act)
        torch.cuda.synchronize()
        U.assert_close(C.cpu().numpy(), ref, what=f"bias_act {act} pad {pad}")


def test_unfused_pieces():
    M, N = 333, 1031
    announce("pointwise")
    C0 = D.uniform_f16(90, (M, N), -4, 4)
    bias = D.uniform_f16(91, (N,))
    C = torch.from_numpy(C0).cuda()
    gba.bias_add_(C, torch.from_numpy(bias).cuda())
    torch.cuda.synchronize()
    want = (C0.astype(np.float32) + bias.astype(np.float32)).astype(np.float16)
    assert np.array_equal(C.cpu().numpy(), want)
    gba.relu_(C)
    torch.cuda.synchronize()
    assert np.array_equal(C.cpu().numpy(), np.maximum(want, np.float16(0)))

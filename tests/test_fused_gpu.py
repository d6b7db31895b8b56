"""HIP path vs the CPU oracle for the wider idioms of gba_fused_gemm: ReLU
prologue (Listing 4), sum / difference of two products (Listing 5), full or
subtracted bias, Sigmoid and Tanh -- element by element, through the C ABI.

Each case prints its name before touching the GPU.  Inputs come from the
seeded generators in paper_2006_12645_amd.datagen; expected values from
the oracle only.
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
ACT = {"none": O.ACT_NONE, "relu": O.ACT_RELU, "sigmoid": O.ACT_SIGMOID, "tanh": O.ACT_TANH}


def announce(*what):
    print("CASE", *what, flush=True)


@pytest.fixture(autouse=True, scope="module")
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    gba.lib()
    yield


class Problem:
    """Logical operands of one fused request and its oracle."""

    def __init__(self, seed, M, N, K, K2=None, dist="uniform", bias="row", full_bias=False):
        self.M, self.N, self.K, self.K2 = M, N, K, K2
        self.A, self.B, row = D.random_problem(seed, M, N, K, dist)
        self.P = self.Q = None
        if K2 is not None:
            self.P, self.Q, _ = D.random_problem(seed + 50, M, N, K2, dist)
        if bias is None:
            self.bias = None
        elif full_bias:
            lo, hi = (-8, 8) if dist == "int" else (-1, 1)
            self.bias = (D.integer_f16(seed + 60, (M, N), lo, hi) if dist == "int"
                         else D.uniform_f16(seed + 60, (M, N), lo, hi))
        else:
            self.bias = row

    def oracle(self, prologue=False, second="add", bias_op="add", act="relu", rows=None, acc16=False):
        sec = 0 if self.P is None else (1 if second == "add" else -1)
        return O.fused(D.store(self.A, D.ROW), D.ROW, D.store(self.B, D.COL), D.COL,
                       self.M, self.N, self.K, prologue_relu=prologue, second=sec,
                       p_store=None if self.P is None else D.store(self.P, D.ROW),
                       q_store=None if self.Q is None else D.store(self.Q, D.COL),
                       K2=self.K2 or 0, bias=self.bias, bias_sign=1 if bias_op == "add" else -1,
                       act=ACT[act], rows=rows, acc16=acc16)

    def gpu(self, layout, prologue=False, second="add", bias_op="add", act="relu", accum="f32",
            tile=None, pad=0, offset=False, ld=None, out=None, **extra):
        la, lb = D.LAYOUT_NAMES[layout]

        def dev(x, lay):
            if x is None:
                return None
            if ld is not None:
                # every operand with leading dimension ld, built on the device
                # (NaN padding, as in datagen.store)
                rows, cols = x.shape
                outer, inner = (rows, cols) if lay == D.ROW else (cols, rows)
                t = torch.full((outer, ld), float("nan"), dtype=torch.float16, device="cuda")
                t[:, :inner].copy_(torch.from_numpy(D.store(x, lay)).cuda())
                return t[:, :cols] if lay == D.ROW else t[:, :rows].t()
            if not offset:
                return U.device_operand(x, lay, pad)
            # storage shifted by one element: 2-byte aligned only (general path)
            rows, cols = x.shape
            ext = (cols if lay == D.ROW else rows) + pad
            st = D.store(x, lay, ext)
            flat = torch.empty(st.size + 1, dtype=torch.float16, device="cuda")
            t = flat[1:].view(st.shape)
            t.copy_(torch.from_numpy(st).cuda())
            return t[:, :cols] if lay == D.ROW else t[:, :rows].t()

        dbias = None
        if self.bias is not None:
            dbias = (torch.from_numpy(self.bias).cuda() if self.bias.ndim == 1
                     else dev(self.bias, D.ROW))
        o = gba.fused_gemm(dev(self.A, la), dev(self.B, lb), P=dev(self.P, la), Q=dev(self.Q, lb),
                           second=second, prologue="relu" if prologue else None, bias=dbias,
                           bias_op=bias_op, act=act, accum=accum, tile=tile, out=out, **extra)
        torch.cuda.synchronize()
        return o.cpu().numpy()


# ----------------------------------------------------------------------------
@pytest.mark.parametrize("layout", LAYOUTS)
def test_single_column_left_operand_with_a_second_product(layout):
    """K = 1 makes A a single column (and B a single row), which fits
    either layout: the binding takes the layout of P (and Q) for it."""
    announce("K=1 with a second product", layout)
    pr = Problem(707, 48, 312, 1, K2=456)
    U.assert_close(pr.gpu(layout, second="add", act="sigmoid"), pr.oracle(second="add", act="sigmoid"),
                   what=f"K=1 {layout}")


def test_earlier_runtime_failure_does_not_fail_a_launch():
    """A failed runtime call made earlier on the same thread (hipSetDevice
    with a device index that does not exist: rejected on the host, nothing
    reaches the GPU) leaves the thread's last error set; the library's
    launches must neither report it as their own nor skip their work, and
    they leave it cleared.  The operands are on the device before the
    failed call, so that only the library runs between it and the check."""
    import ctypes
    announce("stale runtime error")
    hip = gba.lib()  # resolves the runtime's own symbols through the library's dependencies
    hip.hipSetDevice.argtypes = [ctypes.c_int]
    hip.hipSetDevice.restype = ctypes.c_int
    hip.hipGetLastError.restype = ctypes.c_int
    pr = Problem(705, 264, 136, 200)
    A, B = U.device_operand(pr.A, D.ROW), U.device_operand(pr.B, D.COL)
    bias = torch.from_numpy(pr.bias).cuda()
    out = torch.empty((pr.M, pr.N), dtype=torch.float16, device="cuda")
    C = torch.from_numpy(D.uniform_f16(706, (64, 72), -1, 1)).cuda()
    want_relu = np.maximum(C.cpu().numpy(), 0)
    torch.cuda.synchronize()
    assert hip.hipSetDevice(1 << 20) != 0
    gba.fused_gemm(A, B, bias=bias, out=out)
    assert hip.hipGetLastError() == 0
    assert hip.hipSetDevice(1 << 20) != 0
    gba.relu_(C)
    assert hip.hipGetLastError() == 0
    torch.cuda.synchronize()
    U.assert_close(out.cpu().numpy(), pr.oracle(), what="fused after a failed runtime call")
    assert np.array_equal(C.cpu().numpy(), want_relu)


# Each idiom in all layouts, several tiles plus a ragged tail on the fast path

@pytest.mark.parametrize("layout", LAYOUTS)
def test_prologue_relu(layout):
    announce("prologue_relu", layout)
    pr = Problem(700, 520, 392, 264)
    U.assert_close(pr.gpu(layout, prologue=True), pr.oracle(prologue=True), what=f"prologue {layout}")


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("second", ["add", "sub"])
def test_sum_of_products(layout, second):
    announce("sum_of_products", layout, second)
    pr = Problem(710, 520, 392, 264, K2=136)
    U.assert_close(pr.gpu(layout, second=second), pr.oracle(second=second),
                   what=f"second {second} {layout}")


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("bias_op", ["add", "sub"])
def test_full_bias(layout, bias_op):
    announce("full_bias", layout, bias_op)
    pr = Problem(720, 264, 392, 200, full_bias=True)
    U.assert_close(pr.gpu(layout, bias_op=bias_op, act="none", pad=8),
                   pr.oracle(bias_op=bias_op, act="none"), what=f"full bias {bias_op} {layout}")


@pytest.mark.parametrize("layout", ["RC", "CR"])
@pytest.mark.parametrize("act", ["sigmoid", "tanh", "none", "relu"])
def test_activations(layout, act):
    announce("activation", layout, act)
    pr = Problem(730, 328, 264, 512, dist="mlp")
    got = pr.gpu(layout, act=act, bias_op="sub")
    ref = pr.oracle(act=act, bias_op="sub")
    U.assert_close(got, ref, what=f"{act} {layout}")
    if act in ("sigmoid", "tanh"):
        # bounded outputs: the error is the fp16 rounding plus a few fp32 ulps
        err = np.abs(got.astype(np.float64) - ref)
        assert err.max() <= 2e-3, err.max()


def test_tanh_small_arguments():
    """Pre-activations spread over [-2^-3, 2^-3]: both sides of the Taylor /
    exponential switch of tanh, against the oracle to fp16 rounding."""
    announce("tanh_small")
    M, N, K = 256, 256, 64
    A = D.uniform_f16(740, (M, K), -1, 1)
    B = D.uniform_f16(741, (K, N), -1 / 64, 1 / 64)
    pr = Problem(742, M, N, K, bias=None)
    pr.A, pr.B = A, B
    got = pr.gpu("RC", act="tanh").astype(np.float64)
    ref = pr.oracle(act="tanh")
    assert np.abs(ref).max() < 0.3 and (np.abs(ref) < 1 / 16).any() and (np.abs(ref) > 1 / 16).any()
    assert (np.abs(got - ref) <= 1e-5 + 2.0 ** -10 * np.abs(ref)).all()


@pytest.mark.parametrize("layout", LAYOUTS)
def test_everything_at_once(layout):
    announce("all_features", layout)
    pr = Problem(750, 392, 520, 200, K2=328, full_bias=True)
    kw = dict(prologue=True, second="sub", bias_op="sub", act="tanh")
    U.assert_close(pr.gpu(layout, **kw, pad=16), pr.oracle(**kw), what=f"all {layout}")


# ----------------------------------------------------------------------------
# Every tile, and fp16 accumulation

@pytest.mark.parametrize("tile", range(NUM_TILES))
@pytest.mark.parametrize("layout", LAYOUTS)
def test_every_tile_all_features(tile, layout):
    announce("tile all features", tile, layout)
    pr = Problem(760, 520, 392, 264, K2=200, full_bias=True)
    kw = dict(prologue=True, second="sub", bias_op="add", act="relu")
    U.assert_close(pr.gpu(layout, **kw, tile=tile), pr.oracle(**kw), what=f"tile {tile} {layout}")


@pytest.mark.parametrize("tile", [1, 16, 17, 18, 19, 20])
@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("accum", ["f32", "f16"])
def test_prologue_on_eight_wave_tiles(tile, layout, accum):
    """The prologue ReLU on the 8-wave tiles, one product: on some of them
    (row-major A) the A fragments are rectified as they are read and the
    left tile arrives by direct copies, on the others the left tile is
    staged through registers; both must give the oracle's result."""
    announce("prologue 8-wave", tile, layout, accum)
    pr = Problem(1000 + tile, 264, 328, 200, bias="row")
    U.assert_close(pr.gpu(layout, prologue=True, accum=accum, tile=tile), pr.oracle(prologue=True, acc16=accum == "f16"),
                   accum=accum, what=f"prologue tile {tile} {layout} {accum}")


@pytest.mark.parametrize("tile", [1, 4, 6, 9])
@pytest.mark.parametrize("layout", ["RC", "CR"])
def test_fp16_accumulation_two_products(tile, layout):
    announce("f16acc", tile, layout)
    pr = Problem(770, 264, 392, 256, K2=128)
    kw = dict(prologue=True, second="add", act="relu")
    U.assert_close(pr.gpu(layout, **kw, accum="f16", tile=tile), pr.oracle(**kw), accum="f16",
                   what=f"f16 tile {tile} {layout}")


def ulp16(x):
    """Spacing of binary16 values at magnitude |x| (subnormal spacing below
    2^-14)."""
    e = np.floor(np.log2(np.maximum(np.abs(x), 2.0 ** -14)))
    return 2.0 ** (e - 10)


@pytest.mark.parametrize("tile", [1, 4, 6, 9, None])
@pytest.mark.parametrize("layout", ["RC", "CR", "RR", "CC"])
def test_fp16_accumulation_matches_its_emulation(tile, layout):
    """fp16 accumulation against the oracle's emulation of the reading (the
    running sum rounded to binary16 after every aligned group of 32 k).  The
    GPU sums each group in fp32 in the MFMA's own order, so a group-end
    rounding can land on the other side of a tie: allow one binary16 step of
    the running sum, and require almost every output to agree to the output
    rounding alone."""
    announce("f16acc_emulation", tile, layout)
    pr = Problem(860, 264, 328, 1000, K2=200, bias="row")
    kw = dict(prologue=True, second="sub", act="none")
    got = pr.gpu(layout, accum="f16", tile=tile, **kw).astype(np.float64)
    emu = pr.oracle(acc16=True, **kw)
    err = np.abs(got - emu)
    assert (err <= 2 * ulp16(np.maximum(np.abs(emu), 64.0))).all(), err.max()
    close = err <= 0.5 * ulp16(emu) + 1e-12
    assert close.mean() >= 0.99, close.mean()


# The four-stage small tiles that run with copy-only waves: 21-25 in RC, the
# 32x128 one in RR and the 128x32 one in CC.
COPY_WAVE_TILES = [(21, "RC"), (22, "RC"), (23, "RC"), (24, "RC"), (25, "RC"), (24, "RR"), (25, "CC")]


@pytest.mark.parametrize("tile,layout", COPY_WAVE_TILES)
@pytest.mark.parametrize("second", [None, "add", "sub"])
def test_fp16_accumulation_small_tiles_match_emulation(tile, layout, second):
    """The four-stage small tiles keep the fp16 running sum as fp16 and add
    each 32-deep group's own fp32 sum to it (one rounding per group), where
    both operand tiles arrive by direct copies and without a prologue: held
    to the oracle's emulation of the reading as the other tiles are, and
    bit-exact on integer data."""
    announce("f16acc small tile", tile, layout, second)
    kw = dict(act="none") if second is None else dict(second=second, act="none")
    K2 = None if second is None else 200
    pr = Problem(870 + tile, 264, 328, 1000, K2=K2, bias="row")
    got = pr.gpu(layout, accum="f16", tile=tile, **kw).astype(np.float64)
    emu = pr.oracle(acc16=True, **kw)
    err = np.abs(got - emu)
    assert (err <= 2 * ulp16(np.maximum(np.abs(emu), 64.0))).all(), err.max()
    close = err <= 0.5 * ulp16(emu) + 1e-12
    assert close.mean() >= 0.99, close.mean()
    pri = Problem(880 + tile, 264, 328, 392, K2=None if second is None else 136, dist="int", full_bias=True)
    kwi = dict(act="relu") if second is None else dict(second=second, act="relu")
    got = pri.gpu(layout, accum="f16", tile=tile, **kwi)
    assert np.array_equal(got.astype(np.float64), pri.oracle(**kwi)), "integer data not exact"


@pytest.mark.parametrize("tile,layout", COPY_WAVE_TILES)
@pytest.mark.parametrize("accum", ["f32", "f16"])
@pytest.mark.parametrize("K,K2", [(8, None), (64, None), (136, None), (256, None), (328, None), (40, 72),
                                  (256, 8), (0, 64), (64, 0), (0, 0)])
def test_copy_wave_small_tiles_step_counts(tile, layout, accum, K, K2):
    """Reductions of one step, of fewer steps than the four LDS stages, of
    exactly four and of more, and empty ones, in one and in two products, on
    the small tiles whose copies are issued by waves that do not compute:
    each step's barrier must pair up between the two kinds of waves, and
    the copies past the last step must stay out of the result."""
    announce("copy-wave small tile steps", tile, layout, accum, K, K2)
    kw = dict(act="none") if K2 is None else dict(second="sub", act="none")
    pr = Problem(900 + tile + K, 96, 160, K, K2=K2, bias="row")
    got = pr.gpu(layout, accum=accum, tile=tile, **kw).astype(np.float64)
    if accum == "f16":
        emu = pr.oracle(acc16=True, **kw)
        err = np.abs(got - emu)
        assert (err <= 2 * ulp16(np.maximum(np.abs(emu), 64.0))).all(), err.max()
    else:
        U.assert_close(got, pr.oracle(**kw), what=f"steps tile {tile} {layout} K={K} K2={K2}")
    pri = Problem(950 + tile + K, 96, 160, K, K2=K2, dist="int", full_bias=True)
    kwi = dict(act="relu") if K2 is None else dict(second="add", act="relu")
    got = pri.gpu(layout, accum=accum, tile=tile, **kwi)
    assert np.array_equal(got.astype(np.float64), pri.oracle(**kwi)), "integer data not exact"


@pytest.mark.parametrize("tile", [None, 1, 4, 6, 9, 18, 19, 20, 21, 22, 23, 24, 25, "general"])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_fp16_accumulation_sum_of_products_golden(tile, layout):
    """The hand-derived binary16 results of the single running sum through
    A.B and then P.Q (tests/golden/acc16_sum_of_products.json), chosen so
    that two separate accumulators would give another value.  Each golden
    row of A and P sits in the first and last row of a 264x264 problem and B
    and Q have ones in the first and last column, so the four corner outputs
    carry the golden value (including shifted edge tiles) and every other
    output is 0."""
    import oracle_pins_acc16 as PA
    M = N = 264
    for case in PA.golden_acc16_sum_of_products():
        announce("f16acc golden", case["name"], tile, layout)
        K, K2 = case["K"], case["K2"]
        pr = Problem(0, M, N, K, K2=K2, bias=None)
        pr.A, pr.P = np.zeros((M, K), np.float16), np.zeros((M, K2), np.float16)
        pr.B, pr.Q = np.zeros((K, N), np.float16), np.zeros((K2, N), np.float16)
        for r in (0, M - 1):
            pr.A[r] = PA.golden_row(case["A"], K)[0]
            pr.P[r] = PA.golden_row(case["P"], K2)[0]
        for c in (0, N - 1):
            pr.B[:, c] = 1
            pr.Q[:, c] = 1
        second = "add" if case["second"] > 0 else "sub"
        kw = dict(second=second, act="none", accum="f16")
        if tile == "general":
            got = pr.gpu(layout, offset=True, **kw)
        else:
            got = pr.gpu(layout, tile=tile, **kw)
        want = np.zeros((M, N))
        for r in (0, M - 1):
            for c in (0, N - 1):
                want[r, c] = case["one_sum"]
        assert np.array_equal(got.astype(np.float64), want), (case["name"], got[0, 0], got[-1, -1])


# ----------------------------------------------------------------------------
# Integer data: every partial sum is a small integer, so results are exact

@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("accum", ["f32", "f16"])
@pytest.mark.parametrize("second", ["add", "sub"])
def test_integer_exact(layout, accum, second):
    announce("integer", layout, accum, second)
    pr = Problem(780, 264, 328, 392, K2=136, dist="int", full_bias=True)
    for kw in (dict(prologue=True, second=second, bias_op="sub", act="none"),
               dict(prologue=False, second=second, bias_op="add", act="relu")):
        got = pr.gpu(layout, accum=accum, **kw).astype(np.float64)
        ref = pr.oracle(**kw)
        assert np.array_equal(got, ref), (kw, np.abs(got - ref).max())


# The 256x256 eight-wave tile runs on 16x16x32 MFMAs for reduction-contiguous
# operands: its own checks, on sizes that shift its edge tiles inside the matrix.

@pytest.mark.parametrize("act", ["sigmoid", "tanh"])
def test_headline_tile_activations(act):
    announce("tile 1 activation", act)
    pr = Problem(731, 600, 536, 328, dist="mlp")
    got = pr.gpu("RC", act=act, bias_op="sub", tile=1)
    ref = pr.oracle(act=act, bias_op="sub")
    U.assert_close(got, ref, what=f"tile 1 {act}")
    assert np.abs(got.astype(np.float64) - ref).max() <= 2e-3


@pytest.mark.parametrize("accum", ["f32", "f16"])
def test_headline_tile_integer_exact(accum):
    announce("tile 1 integer", accum)
    pr = Problem(781, 600, 536, 392, K2=136, dist="int", full_bias=True)
    for kw in (dict(prologue=True, second="sub", bias_op="sub", act="none"),
               dict(prologue=False, second="add", bias_op="add", act="relu")):
        got = pr.gpu("RC", accum=accum, tile=1, **kw).astype(np.float64)
        ref = pr.oracle(**kw)
        assert np.array_equal(got, ref), (kw, np.abs(got - ref).max())


# Large shapes on the 8-wave tiles: more output tiles than compute units (two
# or more rounds of workgroups), ragged edges and a K tail; every output
# against the oracle.

@pytest.mark.parametrize("tile,M,N", [(1, 4168, 5160), (16, 4104, 4136), (17, 4104, 4136),
                                      (18, 4168, 3112), (19, 4168, 3112), (20, 4168, 3112)])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_large_shapes_on_eight_wave_tiles(tile, M, N, layout):
    announce("large 8-wave", tile, layout, M, N)
    pr = Problem(790 + tile, M, N, 200, full_bias=tile % 2 == 0)
    kw = dict(prologue=tile % 3 == 0, bias_op="sub" if tile % 2 else "add", act="relu")
    got = pr.gpu(layout, tile=tile, **kw)
    U.assert_close(got, pr.oracle(**kw), what=f"tile {tile} {layout}")


@pytest.mark.parametrize("tile", [4, 10, 13, 14])
def test_integer_exact_split_k(tile):
    announce("integer_splitk", tile)
    pr = Problem(790, 264, 392, 1000, K2=520, dist="int")
    kw = dict(prologue=True, second="sub", act="none")
    got = pr.gpu("RC", tile=tile, **kw).astype(np.float64)
    assert np.array_equal(got, pr.oracle(**kw))


# ----------------------------------------------------------------------------
# Edge cases: empty reductions, small and ragged shapes, the general path

@pytest.mark.parametrize("K,K2", [(0, 64), (64, 0), (0, 0), (8, 8), (1000, 24)])
def test_empty_and_short_reductions(K, K2):
    announce("short_reductions", K, K2)
    pr = Problem(800, 264, 256, K, K2=K2)
    kw = dict(prologue=True, second="sub", act="relu")
    U.assert_close(pr.gpu("RC", **kw), pr.oracle(**kw), what=f"K={K} K2={K2}")


@pytest.mark.parametrize("shape", [(1, 1, 1, 1), (7, 13, 5, 9), (33, 65, 17, 3), (100, 36, 70, 130)])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_general_path_sizes(shape, layout):
    M, N, K, K2 = shape
    announce("general_sizes", shape, layout)
    pr = Problem(810, M, N, K, K2=K2, full_bias=True)
    kw = dict(prologue=True, second="add", bias_op="sub", act="sigmoid")
    U.assert_close(pr.gpu(layout, **kw), pr.oracle(**kw), what=f"{shape} {layout}")


@pytest.mark.parametrize("layout", LAYOUTS)
def test_unaligned_operands_general_path(layout):
    announce("unaligned", layout)
    pr = Problem(820, 200, 136, 72, K2=40, full_bias=True)
    kw = dict(prologue=True, second="sub", bias_op="add", act="tanh")
    U.assert_close(pr.gpu(layout, **kw, offset=True, pad=3), pr.oracle(**kw),
                   what=f"unaligned {layout}")


# The fast path addresses each operand tile with 32-bit offsets and so takes
# leading dimensions below 2^21 elements; larger ones go to the general path.
# Both sides of that limit, every operand (and the full bias) at that leading
# dimension, the output at a leading dimension above it.
FAST_MAX_LD = 1 << 21


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("ld", [FAST_MAX_LD - 8, FAST_MAX_LD])
def test_large_leading_dimensions(layout, ld):
    pr = Problem(830, 300, 264, 264, K2=136, full_bias=True)
    kw = dict(prologue=True, second="sub", bias_op="sub", act="relu")
    ref = pr.oracle(**kw)
    big = torch.full((pr.M, FAST_MAX_LD + 8), float("nan"), dtype=torch.float16, device="cuda")
    out = big[:, :pr.N]
    for tile in (None, 1, 11):
        announce("large_ld", layout, ld, tile)
        U.assert_close(pr.gpu(layout, **kw, tile=tile, ld=ld, out=out), ref,
                       what=f"ld={ld} {layout} tile {tile}")
        # the output's padding stays untouched
        assert torch.isnan(big[:, pr.N:pr.N + 64]).all().item()
    del big, out
    torch.cuda.empty_cache()


@pytest.mark.parametrize("tile,layout", COPY_WAVE_TILES)
@pytest.mark.parametrize("ld", [FAST_MAX_LD - 8, FAST_MAX_LD])
def test_large_leading_dimensions_copy_wave_tiles(tile, layout, ld):
    """The small tiles whose copies run on waves of their own (no prologue),
    with both products at the fast path's largest leading dimension and
    just past it."""
    pr = Problem(835, 300, 264, 264, K2=136, full_bias=True)
    kw = dict(second="sub", bias_op="sub", act="relu")
    ref = pr.oracle(**kw)
    big = torch.full((pr.M, FAST_MAX_LD + 8), float("nan"), dtype=torch.float16, device="cuda")
    out = big[:, :pr.N]
    announce("large_ld copy waves", tile, layout, ld)
    U.assert_close(pr.gpu(layout, **kw, tile=tile, ld=ld, out=out), ref, what=f"ld={ld} {layout} tile {tile}")
    assert torch.isnan(big[:, pr.N:pr.N + 64]).all().item()
    del big, out
    torch.cuda.empty_cache()


# ----------------------------------------------------------------------------
# Reduction split across workgroups (partials in a workspace, summed by the
# last split of each tile)

def split_workspace(nbytes=64 << 20):
    return torch.zeros(nbytes, dtype=torch.uint8, device="cuda")


def counters_zero(ws, tile, M, N):
    """The per-tile counters at the start of the workspace are back at 0."""
    info = gba.tile_info(tile)
    tiles = -(-M // info["bm"]) * -(-N // info["bn"])
    return not ws[:tiles * 4].any().item()


@pytest.mark.parametrize("tile", [4, 5, 6, 7, 8, 9, 18, 19, 20, 21, 22, 23, 24, 25])
@pytest.mark.parametrize("split", [2, 3, 7])
def test_split_reduction_all_features(tile, split):
    # 16 + 4 steps of A.B and P.Q, ragged output (shifted edge tiles)
    announce("split", tile, split)
    pr = Problem(840, 300, 264, 1000, K2=200, full_bias=True)
    kw = dict(prologue=True, second="sub", bias_op="sub", act="tanh")
    ws = split_workspace()
    U.assert_close(pr.gpu("RC", **kw, tile=tile, split=split, workspace=ws), pr.oracle(**kw),
                   what=f"tile {tile} split {split}")
    assert counters_zero(ws, tile, 300, 264), "split counters not reset"


@pytest.mark.parametrize("layout", LAYOUTS)
def test_split_reduction_layouts(layout):
    announce("split_layouts", layout)
    pr = Problem(841, 256, 320, 704, K2=136)
    kw = dict(prologue=False, second="add", act="relu")
    U.assert_close(pr.gpu(layout, **kw, tile=6, split=4, workspace=split_workspace()), pr.oracle(**kw),
                   what=f"split {layout}")


@pytest.mark.parametrize("split", [2, 3, 5, 16])
def test_split_integer_exact(split):
    announce("split_int", split)
    pr = Problem(842, 200, 136, 1024, K2=64, dist="int")
    kw = dict(second="sub", act="none")
    got = pr.gpu("RC", **kw, tile=6, split=split, workspace=split_workspace())
    assert np.array_equal(got.astype(np.float64), pr.oracle(**kw))


def test_split_deterministic_and_reusable():
    announce("split_repeat")
    pr = Problem(843, 512, 512, 2048)
    ws = split_workspace()
    first = pr.gpu("RC", tile=4, split=8, workspace=ws)
    for _ in range(3):
        assert np.array_equal(pr.gpu("RC", tile=4, split=8, workspace=ws), first)
    assert counters_zero(ws, 4, 512, 512)
    U.assert_close(first, pr.oracle(), what="split 8")


@pytest.mark.parametrize("tile", [None, 4, 6, 9])
def test_mn_contiguous_operands_all_features_odd_k(tile):
    # column-major A and P, row-major B and Q: fast path with K and K2 odd,
    # prologue on the transposed fragments, difference of products, full bias
    announce("CR all features odd K", tile)
    pr = Problem(849, 200, 136, 333, K2=71, full_bias=True)
    kw = dict(prologue=True, second="sub", bias_op="sub", act="sigmoid")
    U.assert_close(pr.gpu("CR", **kw, tile=tile), pr.oracle(**kw), what=f"CR odd K tile {tile}")


def test_split_workspace_reused_with_new_data():
    # a second problem through the same workspace reads its own partials,
    # not the first one's
    announce("split_reuse")
    ws = split_workspace()
    first, second = Problem(846, 256, 192, 1536), Problem(847, 256, 192, 1536)
    first.gpu("RC", tile=6, split=6, workspace=ws)
    U.assert_close(second.gpu("RC", tile=6, split=6, workspace=ws), second.oracle(), what="reuse")
    assert counters_zero(ws, 6, 256, 192)


def test_split_workspace_shared_by_different_tile_counts():
    """Calls with different numbers of output tiles share one workspace: a
    call with few tiles keeps partials where a later call with more tiles
    keeps counters, so every call must leave all the bytes it used at zero
    (a regression: the partials used to stay behind and corrupt the next
    call's arrival counts).  Each call against the oracle, and the whole
    workspace back at zero after each."""
    ws = split_workspace(8 << 20)
    for tile, M, N, K in [(9, 248, 352, 168), (21, 248, 352, 1000), (22, 136, 200, 520),
                          (23, 248, 352, 168), (6, 200, 136, 2000), (9, 248, 352, 168)]:
        announce("split shared ws", tile, M, N, K)
        pr = Problem(845 + tile, M, N, K, K2=72)
        kw = dict(prologue=True, second="sub", act="none")
        U.assert_close(pr.gpu("RC", **kw, tile=tile, split=2, workspace=ws), pr.oracle(**kw),
                       what=f"tile {tile} shared workspace")
        assert not ws.any().item(), f"tile {tile} left non-zero bytes in the workspace"


def test_library_split_on_long_reduction():
    # 64 x 512 outputs over K = 32768: the library splits each 64x64 tile's
    # reduction 16 ways when given a workspace, and runs unsplit without one
    announce("library_split")
    pr = Problem(848, 64, 512, 32768)
    ref = pr.oracle()
    U.assert_close(pr.gpu("RC"), ref, what="auto split")
    U.assert_close(pr.gpu("RC", workspace=None), ref, what="no workspace")


def test_split_needs_a_workspace():
    # without a workspace (or with split 1) the call runs unsplit: same
    # bits as the unsplit kernel
    announce("split_no_ws")
    pr = Problem(844, 256, 256, 512)
    plain = pr.gpu("RC", tile=6, split=1)
    assert np.array_equal(pr.gpu("RC", tile=6, split=4, workspace=None), plain)
    split = pr.gpu("RC", tile=6, split=4, workspace=split_workspace())
    U.assert_close(split, pr.oracle(), what="split 4")


def test_gemm_bias_act_is_the_single_product_case():
    """gemm_bias_act and gba_fused_gemm with one product and a row bias run
    the same kernel: bitwise equal outputs."""
    announce("single_product_equivalence")
    pr = Problem(830, 520, 392, 264)
    dA = U.device_operand(pr.A, D.ROW)
    dB = U.device_operand(pr.B, D.COL)
    dbias = torch.from_numpy(pr.bias).cuda()
    a = gba.gemm_bias_act(dA, dB, dbias, act="relu")
    b = gba.fused_gemm(dA, dB, bias=dbias, act="relu")
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_deterministic():
    announce("deterministic")
    pr = Problem(840, 520, 392, 264, K2=200, full_bias=True)
    kw = dict(prologue=True, second="sub", act="tanh")
    first = pr.gpu("RC", **kw)
    for _ in range(2):
        assert np.array_equal(pr.gpu("RC", **kw), first)


def test_sum4096_full():
    """The sum-of-products workload at full size (4096^3 twice), every output
    against the oracle, in the launch the benchmark times."""
    w = D.WORKLOADS["sum4096_RC"]
    announce(w.name, "every output")
    A, B, bias = D.logical_inputs(w)
    P, Q = D.second_inputs(w)
    dA = U.device_operand(A, D.ROW)
    dB = U.device_operand(B, D.COL)
    dP = U.device_operand(P, D.ROW)
    dQ = U.device_operand(Q, D.COL)
    out = gba.fused_gemm(dA, dB, P=dP, Q=dQ, bias=torch.from_numpy(bias).cuda(), act="relu")
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    ref = O.fused(D.store(A, D.ROW), D.ROW, D.store(B, D.COL), D.COL, w.M, w.N, w.K, second=1,
                  p_store=D.store(P, D.ROW), q_store=D.store(Q, D.COL), K2=w.extra["K2"], bias=bias,
                  act=O.ACT_RELU)
    U.assert_close(got, ref, what=w.name)


def test_prologue4096_full():
    w = D.WORKLOADS["prologue4096_RC"]
    announce(w.name, "every output")
    A, B, bias = D.logical_inputs(w)
    out = gba.fused_gemm(U.device_operand(A, D.ROW), U.device_operand(B, D.COL), prologue="relu",
                         bias=torch.from_numpy(bias).cuda(), act="relu")
    torch.cuda.synchronize()
    ref = O.fused(D.store(A, D.ROW), D.ROW, D.store(B, D.COL), D.COL, w.M, w.N, w.K,
                  prologue_relu=True, bias=bias, act=O.ACT_RELU)
    U.assert_close(out.cpu().numpy(), ref, what=w.name)


def test_unfused_add_piece():
    """gba_add_f16 (the separate add of the unfused sum-of-matmuls chain):
    the fp32 sum of two fp16 values is exact, so the result is that sum
    rounded once to fp16 -- numpy's float16 addition."""
    announce("unfused_add")
    M, N = 77, 136
    C = D.uniform_f16(850, (M, N), -4, 4)
    X = D.uniform_f16(851, (M, N), -4, 4)
    dC = U.device_operand(C, D.ROW, pad=8)
    dX = U.device_operand(X, D.ROW, pad=0)
    gba.add_(dC, dX)
    torch.cuda.synchronize()
    want = (C.astype(np.float32) + X.astype(np.float32)).astype(np.float16)
    assert np.array_equal(dC.cpu().numpy(), want)
    dC2 = U.device_operand(C, D.ROW)[:, 1:]      # 2-byte aligned view: scalar path
    dX2 = U.device_operand(X, D.ROW)[:, 1:]
    gba.add_(dC2, dX2)
    torch.cuda.synchronize()
    assert np.array_equal(dC2.cpu().numpy(), want[:, 1:])

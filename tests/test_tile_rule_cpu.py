"""The library's tile choice, through its host-only queries (no GPU).

gba_fused_tile reports the tile gba_fused_gemm would run a request on.
Without the prologue that is gba_select_tile's choice for the total
reduction length; with it, the tiles whose copies are issued by waves of
their own (which they have only without the prologue) are never taken.  The
pinned cases are measured choices: each names the times it rests on (MI355X,
warm / with operands from HBM, microseconds)."""
import ctypes
import random

import pytest

from paper_2006_12645_amd import gba

FAKE = 0x10000  # 16-byte aligned, never dereferenced: these queries do not touch memory
LAYOUTS = {"RR": (0, 0), "RC": (0, 1), "CR": (1, 0), "CC": (1, 1)}
ACCS = {"f32": gba.GBA_ACC_F32, "f16": gba.GBA_ACC_F16}


def desc(M, N, K, layout="RC", accum="f32", prologue=False, K2=0, tile=-1):
    la, lb = LAYOUTS[layout]
    d = gba.new_desc()
    d.layoutA, d.layoutB, d.M, d.N, d.K = la, lb, M, N, K
    d.A, d.lda = FAKE, (K if la == 0 else M)
    d.B, d.ldb = FAKE, (N if lb == 0 else K)
    if K2:
        d.second, d.K2 = gba.GBA_SECOND_ADD, K2
        d.P, d.ldp = FAKE, (K2 if la == 0 else M)
        d.Q, d.ldq = FAKE, (N if lb == 0 else K2)
    d.prologue = gba.GBA_PRO_RELU if prologue else gba.GBA_PRO_NONE
    d.bias_kind, d.bias = gba.GBA_BIAS_ROW, FAKE
    d.act, d.C, d.ldc = gba.GBA_ACT_RELU, FAKE, N
    d.accum = ACCS[accum]
    d.tile_id = tile
    return d


def shapes(seed, n):
    rng = random.Random(seed)
    dims = [32, 64, 96, 128, 256, 384, 512, 640, 1000, 1024, 1536, 2048, 3072, 4096, 8192]
    return [(rng.choice(dims), rng.choice(dims), rng.choice(dims[1:])) for _ in range(n)]


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("accum", ACCS)
def test_fused_tile_without_prologue_is_select_tile(layout, accum):
    la, lb = LAYOUTS[layout]
    for M, N, K in shapes(11, 300):
        for K2 in (0, K // 16 * 8):  # a second reduction that keeps the fast path's 8-element alignment
            want = gba.select_tile(M, N, K + K2, la, lb, accum=accum)
            assert gba.fused_tile(desc(M, N, K, layout, accum, K2=K2)) == want, (M, N, K, K2)


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("accum", ACCS)
def test_prologue_never_takes_copy_wave_tiles(layout, accum):
    """Tiles 24 / 25 (and, with fp32 accumulation, 21 / 23) run their copies
    on waves of their own only without the prologue; with it they were the
    slowest of the small tiles, so the rule does not give them a request
    with the prologue."""
    banned = {24, 25} | ({21, 23} if accum == "f32" or layout == "CR" else set())
    for M, N, K in shapes(12, 300):
        t = gba.fused_tile(desc(M, N, K, layout, accum, prologue=True))
        assert t not in banned or (layout == "RC" and accum == "f16"), (M, N, K, t)


@pytest.mark.parametrize("accum", ACCS)
@pytest.mark.parametrize("prologue", [False, True])
def test_cr_never_takes_four_stage_small_tiles(accum, prologue):
    """In CR no small four-stage tile has copy-only waves (both operand
    tiles are M- or N-contiguous and shorter than 128 elements per row), and
    the two-stage and k-group tiles were faster there."""
    for M, N, K in shapes(13, 300):
        t = gba.fused_tile(desc(M, N, K, "CR", accum, prologue=prologue))
        assert t not in {21, 23, 24, 25}, (M, N, K, t)


@pytest.mark.parametrize("case,tile", [
    # fp32 1024^3, RR: 32x128 four-stage tile 7.84 / 8.43 against 8.78 / 10.95
    # on 64x64 with two k-groups; with the prologue (no copy-only waves)
    # 64x64 with four k-groups 9.19 / 11.60 against 12.17 / 15.38 on 32x128
    (dict(M=1024, N=1024, K=1024, layout="RR"), 24),
    (dict(M=1024, N=1024, K=1024, layout="RR", prologue=True), 10),
    # CC: the 128x32 tile 7.48 / 8.39 against 8.74 / 10.80; with the
    # prologue 64x64 with four k-groups 9.46 / 11.59
    (dict(M=1024, N=1024, K=1024, layout="CC"), 25),
    (dict(M=1024, N=1024, K=1024, layout="CC", prologue=True), 10),
    # fp16 accumulation, RR: 32x128 11.89 / 12.30 against 10.61 / 16.62 on
    # the 8-wave 64x128 tile; with the prologue the 8-wave tile, 11.38 /
    # 15.72 against 18.25 / 19.28
    (dict(M=1024, N=1024, K=1024, layout="RR", accum="f16"), 24),
    (dict(M=1024, N=1024, K=1024, layout="RR", accum="f16", prologue=True), 20),
    # fp16 accumulation, 192 256x256 tiles: 8-wave 128x128 131.1 / 138.1
    # against 140.5 / 139.9 on 256x256 (RC, K = 4096); at 256 of them the
    # 256x256 tile, 172.4 / 162.7 against 170.3 / 176.6
    (dict(M=4096, N=3072, K=4096, accum="f16"), 18),
    (dict(M=4096, N=4096, K=4096, accum="f16"), 1),
    # CR, fp32: 64x64 with four k-groups on 1024^3, 9.09 / 11.38 against
    # 9.19 / 11.81 with two; 128 x 4096 x 2048 on 32x64 with four k-groups
    # 12.29 / 16.88 against 13.10 / 22.74 on 64x64 with two
    (dict(M=1024, N=1024, K=1024, layout="CR"), 10),
    (dict(M=128, N=4096, K=2048, layout="CR"), 12),
    # CR, fp16: 32 x 4096 x 1024 on the two-stage 32x32 tile 10.71 / 16.89
    # against 11.54 / 17.12 on the four-stage one; 1280 x 2816 x 3968 on the
    # 8-wave 64x128 tile 57.82 / 64.32 against 62.62 / 72.91 on 128x128
    (dict(M=32, N=4096, K=1024, layout="CR", accum="f16"), 9),
    (dict(M=1280, N=2816, K=3968, layout="CR", accum="f16"), 20),
    # RC, fp32, 64 x 4096 x 2048 (128 32x64 tiles): 32x32 with four
    # k-groups 7.58 / 9.07 against 7.38 / 10.58 on the four-stage 32x32 tile
    (dict(M=64, N=4096, K=2048), 13),
    (dict(M=64, N=4096, K=1024), 23),
    # short reductions: RR 3072 x 3072 x 128 on the 4-wave 128x128 tile
    # 13.1 / 12.8 against 16.8 / 16.4 on 256x256 (128x64: 12.1 / 11.9; the
    # branch's 384-workgroup limit for 128x128 was the best single limit
    # over the 48 shapes); RC 3200 x 2944 x 128 on the 8-wave 128x128 tile
    # 11.9 / 11.3 against 12.5 / 12.3; 4096^2 x 128 stays on 256x256
    (dict(M=3072, N=3072, K=128, layout="RR"), 4),
    (dict(M=3200, N=2944, K=128), 18),
    (dict(M=4096, N=4096, K=128), 1),
    # a requested tile that fits is kept
    (dict(M=1024, N=1024, K=1024, layout="RR", prologue=True, tile=24), 24),
])
def test_measured_choices(case, tile):
    assert gba.fused_tile(desc(**case)) == tile


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("accum", ACCS)
def test_select_tile_with_prologue_is_fused_tile(layout, accum):
    la, lb = LAYOUTS[layout]
    for M, N, K in shapes(14, 200):
        for pro in (False, True):
            want = gba.fused_tile(desc(M, N, K, layout, accum, prologue=pro))
            assert gba.select_tile(M, N, K, la, lb, accum=accum, prologue=pro) == want, (M, N, K, pro)


def test_fused_tile_errors():
    t = ctypes.c_int(5)
    assert gba.lib().gba_fused_tile(ctypes.byref(desc(64, 64, 64)), None) == gba.GBA_EINVAL
    assert gba.lib().gba_fused_tile(None, ctypes.byref(t)) == gba.GBA_EINVAL
    bad = desc(64, 64, 64)
    bad.act = 9
    assert gba.lib().gba_fused_tile(ctypes.byref(bad), ctypes.byref(t)) == gba.GBA_EINVAL and t.value == -1
    assert gba.fused_tile(desc(0, 64, 64)) == -1

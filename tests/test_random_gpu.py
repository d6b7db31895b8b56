"""Randomised requests through gba_fused_gemm against the oracle: every
combination of layout, tile (or the library's choice), prologue, second
product, bias kind and sign, activation, accumulation, reduction split and
operand alignment, on seeded random shapes that mostly are not multiples of
the tiles.  A second sweep puts every request on one of the 8-wave tiles at
shapes from the tile's size up to ~700 more.  Each case prints its
parameters before touching the GPU.
"""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2006_12645_amd import datagen as D
from paper_2006_12645_amd import gba

import gpu_util as U

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

ACT = {"none": O.ACT_NONE, "relu": O.ACT_RELU, "sigmoid": O.ACT_SIGMOID, "tanh": O.ACT_TANH}
NUM_CASES = 256
NUM_CASES_EIGHT_WAVE = 64


def draw(seed):
    """One random request (plain Python values)."""
    rng = np.random.default_rng(90000 + seed)
    pick = lambda xs: xs[int(rng.integers(len(xs)))]
    # sizes: mostly multiples of 8 (fast path), sometimes not
    mult = 8 if rng.random() < 0.75 else 1
    M = int(rng.integers(1, 50)) * mult + (0 if mult == 8 else int(rng.integers(1, 8)))
    N = int(rng.integers(1, 50)) * mult + (0 if mult == 8 else int(rng.integers(1, 8)))
    K = int(rng.integers(0, 90)) * 8 + (int(rng.integers(0, 8)) if rng.random() < 0.3 else 0)
    c = dict(M=M, N=N, K=K, layout=pick(["RR", "RC", "CR", "CC"]),
             prologue=bool(rng.random() < 0.5), act=pick(list(ACT)),
             accum="f16" if rng.random() < 0.25 else "f32",
             bias=pick([None, "row", "full"]), bias_op=pick(["add", "sub"]),
             second=pick([None, "add", "sub"]), K2=int(rng.integers(0, 60)) * 8,
             offset=bool(rng.random() < 0.1), tile=None, split=None)
    tiles = [t for t in range(gba.num_tiles())
             if gba.tile_info(t)["bm"] <= M and gba.tile_info(t)["bn"] <= N]
    if tiles and rng.random() < 0.6:
        c["tile"] = pick(tiles)
    if c["accum"] == "f32" and rng.random() < 0.3:
        c["split"] = int(rng.integers(2, 9))
    return c


def operand(x, lay, offset):
    """Device tensor of logical matrix x stored in layout lay (leading
    dimension padded by 8); offset: storage shifted by one element."""
    rows, cols = x.shape
    ext = (cols if lay == D.ROW else rows) + 8
    st = D.store(x, lay, ext)
    flat = torch.empty(st.size + 1, dtype=torch.float16, device="cuda")
    t = (flat[1:] if offset else flat[:-1]).view(st.shape)
    t.copy_(torch.from_numpy(st).cuda())
    return t[:, :cols] if lay == D.ROW else t[:, :rows].t()


def draw_eight_wave(seed):
    """A request on one of the 8-wave tiles (the 16x16x32 kernel in most
    layouts), with every dimension at least the tile's and up to ~700 more."""
    c = draw(100000 + seed)
    rng = np.random.default_rng(777000 + seed)
    t = int(rng.choice([1, 16, 17, 18, 19, 20]))
    info = gba.tile_info(t)
    mult = 8 if rng.random() < 0.8 else 1
    c["M"] = info["bm"] + int(rng.integers(0, 700)) // mult * mult + (0 if mult == 8 else int(rng.integers(1, 8)))
    c["N"] = info["bn"] + int(rng.integers(0, 700)) // 8 * 8
    c["tile"] = t
    if c["split"] is not None and info["bm"] * info["bn"] > 128 * 128:
        c["split"] = None
    return c


@pytest.mark.parametrize("seed", range(NUM_CASES))
def test_random_request(seed):
    run_case(seed, draw(seed))


NUM_CASES_LARGE = 96


def draw_large(seed):
    """A request of 128 to 1024 rows and columns and a reduction of up to
    1024 (multiples of 8: the aligned fast path), mostly on the library's
    own tile choice, every other option as in draw()."""
    c = draw(200000 + seed)
    rng = np.random.default_rng(555000 + seed)
    c["M"], c["N"] = int(rng.integers(16, 129)) * 8, int(rng.integers(16, 129)) * 8
    c["K"], c["K2"] = int(rng.integers(1, 129)) * 8, int(rng.integers(0, 65)) * 8
    c["offset"] = False
    c["tile"] = None if rng.random() < 0.8 else int(rng.integers(0, gba.num_tiles()))
    info = gba.tile_info(c["tile"]) if c["tile"] is not None else None
    if info and c["accum"] == "f16" and info["split_k"] > 1:
        c["tile"] = None
    if c["split"] is not None and info and info["bm"] * info["bn"] > 128 * 128:
        c["split"] = None
    return c


@pytest.mark.parametrize("seed", range(NUM_CASES_LARGE))
def test_random_request_large(seed):
    run_case(300000 + seed, draw_large(seed))


@pytest.mark.parametrize("seed", range(NUM_CASES_EIGHT_WAVE))
def test_random_request_eight_wave_tiles(seed):
    run_case(100000 + seed, draw_eight_wave(seed))


def run_case(seed, c):
    print("CASE", seed, c, flush=True)
    M, N, K = c["M"], c["N"], c["K"]
    A, B, _ = D.random_problem(91000 + seed, M, N, K)
    K2 = c["K2"]
    P = Q = None
    if c["second"]:
        P, Q, _ = D.random_problem(92000 + seed, M, N, K2)
    bias = None
    if c["bias"] == "row":
        bias = D.uniform_f16(93000 + seed, (N,))
    elif c["bias"] == "full":
        bias = D.uniform_f16(93000 + seed, (M, N))
    la, lb = D.LAYOUT_NAMES[c["layout"]]
    dev = lambda x, lay: None if x is None else operand(x, lay, c["offset"])
    dbias = None
    if bias is not None:
        dbias = torch.from_numpy(bias).cuda() if bias.ndim == 1 else operand(bias, D.ROW, c["offset"])
    got = gba.fused_gemm(dev(A, la), dev(B, lb), P=dev(P, la), Q=dev(Q, lb), second=c["second"] or "add",
                         prologue="relu" if c["prologue"] else None, bias=dbias, bias_op=c["bias_op"],
                         act=c["act"], accum=c["accum"], tile=c["tile"], split=c["split"])
    torch.cuda.synchronize()
    sec = 0 if P is None else (1 if c["second"] == "add" else -1)
    ref = O.fused(D.store(A, D.ROW), D.ROW, D.store(B, D.COL), D.COL, M, N, K,
                  prologue_relu=c["prologue"], second=sec,
                  p_store=None if P is None else D.store(P, D.ROW),
                  q_store=None if Q is None else D.store(Q, D.COL), K2=K2 if P is not None else 0,
                  bias=bias, bias_kind=(O.BIAS_NONE if bias is None else
                                        O.BIAS_ROW if bias.ndim == 1 else O.BIAS_FULL),
                  bias_sign=1 if c["bias_op"] == "add" else -1, act=ACT[c["act"]],
                  acc16=c["accum"] == "f16")
    U.assert_close(got.cpu().numpy(), ref, accum=c["accum"], what=f"case {seed}")

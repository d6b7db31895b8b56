"""The allocation-free entry point gba_fused_gemm_noalloc (library-held
static scratch) against gba_fused_gemm with a caller-owned workspace: the
same kernels and the same split, so the same bits; and both against the
oracle.  Two calls in a row, the second with a smaller input, so the second
reads the scratch the first one left behind."""
import pytest

from oracle import oracle as O
from paper_2006_12645_amd import datagen as D
from paper_2006_12645_amd import gba

import gpu_util as U

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def announce(*what):
    print("CASE", *what, flush=True)


@pytest.fixture(autouse=True, scope="module")
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    gba.lib()
    yield


def request(seed, M, N, K, K2):
    """Device operands, launch keywords and the oracle of relu(relu(A).B -
    relu(P).Q + bias) (K2 > 0) or relu(A.B + bias) (K2 == 0)."""
    A, B, bias = D.random_problem(seed, M, N, K)
    kw = dict(bias=torch.from_numpy(bias).cuda(), act="relu")
    okw = dict(bias=bias, act=O.ACT_RELU)
    if K2:
        P, Q, _ = D.random_problem(seed + 1, M, N, K2)
        kw.update(P=U.device_operand(P, D.ROW), Q=U.device_operand(Q, D.COL), second="sub", prologue="relu")
        okw.update(second=-1, p_store=D.store(P, D.ROW), q_store=D.store(Q, D.COL), K2=K2, prologue_relu=True)
    ref = O.fused(D.store(A, D.ROW), D.ROW, D.store(B, D.COL), D.COL, M, N, K, **okw)
    return U.device_operand(A, D.ROW), U.device_operand(B, D.COL), kw, ref


# (M, N, K, K2, tile, split): forced splits on two tiles, then the library's
# own choice on a long reduction (64x64 tiles split 16 and 32 ways); each
# pair is a larger then a smaller request
CASES = [
    [(300, 264, 2000, 200, 6, 7), (136, 72, 520, 64, 6, 3)],
    [(392, 520, 1000, 328, 4, 5), (264, 136, 200, 72, 4, 2)],
    [(64, 512, 32768, 0, None, None), (64, 256, 16384, 0, None, None)],
]


@pytest.mark.parametrize("pair", range(len(CASES)))
def test_noalloc_matches_workspace_entry_point(pair):
    ws = torch.zeros(64 << 20, dtype=torch.uint8, device="cuda")
    for (M, N, K, K2, tile, split) in CASES[pair]:
        announce("noalloc", M, N, K, K2, tile, split)
        dA, dB, kw, ref = request(7000 + M + K, M, N, K, K2)
        kw.update(tile=tile, split=split)
        got_static = gba.fused_gemm(dA, dB, workspace="static", **kw)
        got_ws = gba.fused_gemm(dA, dB, workspace=ws, **kw)
        torch.cuda.synchronize()
        assert torch.equal(got_static, got_ws), (M, N, K)
        U.assert_close(got_static.cpu().numpy(), ref, what=f"noalloc {M}x{N}x{K}+{K2}")


def test_noalloc_unsplit_request_uses_no_scratch():
    """A request that does not split runs exactly as gba_fused_gemm."""
    announce("noalloc unsplit")
    dA, dB, kw, ref = request(7100, 520, 392, 264, 136)
    a = gba.fused_gemm(dA, dB, workspace="static", **kw)
    b = gba.fused_gemm(dA, dB, workspace=None, **kw)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    U.assert_close(a.cpu().numpy(), ref, what="noalloc unsplit")

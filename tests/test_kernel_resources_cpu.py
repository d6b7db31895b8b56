"""Register budget of the 16x16x32 kernels, read from the device compiler's
resource report (no GPU needed).

An 8-wave tile of at most 128x128 outputs is sized to run two workgroups per
compute unit: each wave then has at most 128 VGPRs.  A change that pushes
one of these kernels past that budget, or into scratch, halves its
occupancy or adds memory traffic to every step without changing any result,
so the parity tests cannot see it; this test does.  The 256x256 tile runs
one workgroup per compute unit with up to 256 VGPRs per wave; its fp32
one-product kernel in the RC layout (the cube workloads' kernel) must not
spill.
"""
import concurrent.futures as cf
import os
import re
import shutil
import subprocess
import tempfile

import pytest

from paper_2006_12645_amd import build as B


def _have_hipcc():
    try:
        return shutil.which(B._hipcc()) is not None
    except RuntimeError:
        return False


pytestmark = pytest.mark.skipif(not _have_hipcc(), reason="hipcc not available")

NAME = re.compile(r"Function Name: (\S+)")
FIELD = re.compile(r"remark:\s+(VGPRs|ScratchSize \[bytes/lane\]|Occupancy \[waves/SIMD\]): (\d+)")
ARGS = re.compile(r"gemm_bias_act_fast16(I.*)EvNS_8GemmArgsE")


def template_args(mangled):
    """Integer and bool template arguments of a mangled kernel name, in order."""
    m = ARGS.search(mangled)
    return [int(v) for v in re.findall(r"L[ib](-?\d+)E", m.group(1))] if m else None


def resources(unit, tmp):
    src, defines, name = unit
    cmd = ([B._hipcc()] + B.HIPCC_FLAGS + defines +
           ["-Rpass-analysis=kernel-resource-usage", "--cuda-device-only", "-c",
            os.path.join(B.CSRC, src), "-o", os.path.join(tmp, name)])
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    out, cur = {}, None
    for line in r.stderr.splitlines():
        m = NAME.search(line)
        if m:
            cur = out.setdefault(m.group(1), {})
            continue
        m = FIELD.search(line)
        if m and cur is not None:
            cur[m.group(1).split()[0]] = int(m.group(2))
    return out


@pytest.fixture(scope="module")
def fast16_kernels():
    units = [u for u in B.UNITS if u[0] == "gba_gemm_unit.hip"]
    with tempfile.TemporaryDirectory() as tmp, cf.ThreadPoolExecutor(min(8, os.cpu_count() or 1)) as ex:
        reports = list(ex.map(lambda u: resources(u, tmp), units))
    kernels = {}
    for rep in reports:
        for name, res in rep.items():
            args = template_args(name)
            if args is not None:
                kernels[name] = (args, res)
    assert kernels, "no 16x16x32 kernel found in the resource report"
    return kernels


def test_small_eight_wave_tiles_fit_two_workgroups_per_cu(fast16_kernels):
    checked = 0
    for name, (args, res) in fast16_kernels.items():
        bm, bn, wm, wn = args[:4]
        if wm * wn != 8 or bm * bn > 128 * 128:
            continue
        checked += 1
        assert res["ScratchSize"] == 0, (name, res)
        assert res["VGPRs"] <= 128 and res["Occupancy"] >= 4, (name, res)
    assert checked >= 4 * 4 * 3, checked  # three tiles in every layout and variant


def test_four_wave_tiles_do_not_spill(fast16_kernels):
    for name, (args, res) in fast16_kernels.items():
        bm, bn, wm, wn = args[:4]
        if wm * wn < 8:
            assert res["ScratchSize"] == 0, (name, res)


def test_cube_kernel_does_not_spill(fast16_kernels):
    # <256, 256, 2, 4, SK 1, 2 stages, A row-major, B column-major, fp32
    # accumulation, no prologue, one product, not split>
    want = [256, 256, 2, 4, 1, 2, 0, 1, 0, 0, 0, 0]
    hits = [res for args, res in fast16_kernels.values() if args == want]
    assert len(hits) == 1
    assert hits[0]["ScratchSize"] == 0 and hits[0]["Occupancy"] >= 2, hits[0]

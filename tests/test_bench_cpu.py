"""bench.py's host logic on the CPU: the figures it takes from the committed
rocprofv3 summaries are reported only while those summaries were taken on
the current kernel sources, and it refuses more than one GPU."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def _write(path, text):
    with open(path, "w") as f:
        f.write(text)


@pytest.fixture
def profiles(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    return tmp_path


def test_stored_traffic_needs_matching_sources(profiles):
    path = os.path.join(profiles, "gemm_bias_act_cube4096_RC_pmc.md")
    _write(path, f"hbm_bytes_per_launch: 235000000\nkernel_source_sha256: {bench.kernel_source_digest()}\n")
    assert bench.stored_traffic("cube4096_RC") == 235000000.0
    _write(path, "hbm_bytes_per_launch: 235000000\nkernel_source_sha256: " + "0" * 64 + "\n")
    assert bench.stored_traffic("cube4096_RC") is None
    assert bench.stored_traffic("sum4096_RC") is None  # no summary at all


def test_stored_clock_peak_reads_our_kernel_row(profiles):
    path = os.path.join(profiles, f"gemm_bias_act_{bench.HEADLINE}_mfma_util.md")
    rows = ("| kernel | dispatches | MfmaUtil % (median) | GRBM_GUI_ACTIVE (median) | shader clock GHz (median) | "
            "clock-adjusted peak TFLOP/s | rest |\n|---|---|---|---|---|---|---|\n"
            "| `gemm_bias_act_fast16<256, 256, 2, 4, 1, 2, 0, 1, false, false, false, false>` | 20 | 64.6 | "
            "1574712 | 1.876 | 1967 | x |\n"
            "| `hipBLASLt 256x256x64` | 12 | 70.7 | 1441216 | 1.825 | 1914 | x |\n")
    _write(path, rows + f"\nkernel_source_sha256: {bench.kernel_source_digest()}\n")
    assert bench.stored_clock_peak() == (1.876, 1967.0)
    _write(path, rows + "\nkernel_source_sha256: " + "f" * 64 + "\n")
    assert bench.stored_clock_peak() is None


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=300, cwd=ROOT)
    assert r.returncode != 0 and "one GPU" in r.stderr, (r.returncode, r.stderr[-500:])


def test_source_digest_ignores_comments_only():
    src = 'int a = 1; // note\n/* block\n   note */ const char *s = "x // y /* z */";\nint  b;'
    assert bench.strip_comments(src) == 'int a = 1; const char *s = "x // y /* z */"; int b;'
    assert bench.strip_comments(src.replace("note", "other note")) == bench.strip_comments(src)
    assert bench.strip_comments(src.replace("b;", "c;")) != bench.strip_comments(src)

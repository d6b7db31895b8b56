"""Build libgba.so (gfx950 only) in-tree with hipcc.

The entry points (csrc/gba_api.hip) and one kernel-instantiation unit per
operand-layout pair and kernel variant (csrc/gba_gemm_unit.hip compiled with
GBA_LA, GBA_LB, GBA_PRO, GBA_DUAL set) are compiled in parallel, then linked
into ``paper_2006_12645_amd/libgba.so``.  Every hipcc line carries
``-Xclang -target-feature -Xclang -packed-fp32-ops`` so the device compiler
never forms packed fp32 instructions.
"""
import concurrent.futures as cf
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libgba.so")
ARCH = "gfx950"

# (source, extra defines, object name)
UNITS = [("gba_api.hip", [], "gba_api.o")] + [
    ("gba_gemm_unit.hip",
     [f"-DGBA_LA={la}", f"-DGBA_LB={lb}", f"-DGBA_PRO={pro}", f"-DGBA_DUAL={dual}"],
     f"gba_gemm_{'RC'[la]}{'RC'[lb]}_p{pro}d{dual}.o")
    for la in (0, 1) for lb in (0, 1) for pro in (0, 1) for dual in (0, 1)]
HIPCC_FLAGS = ["--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-Wall",
               "-Wno-unused-function", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
               "-I", INCLUDE, "-I", CSRC]


def _hipcc():
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", "hipcc"):
        if c and (os.path.sep not in c or os.path.exists(c)):
            return c
    raise RuntimeError("hipcc not found")


def _compile(unit, verbose):
    src, defines, name = unit
    obj = os.path.join(BUILD, name)
    cmd = [_hipcc()] + HIPCC_FLAGS + defines + ["-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass does not know the packed-fp32 feature name; that warning is expected
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in r.stderr.splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src} {' '.join(defines)}:\n{err}")
    if err.strip() and verbose:
        print(err, flush=True)
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    jobs = max(1, min(len(UNITS), int(os.environ.get("MAX_JOBS", "8"))))
    with cf.ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(lambda u: _compile(u, verbose), UNITS))
    tmp = LIB + ".tmp"
    cmd = [_hipcc(), "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    _check_no_missing_kernels(tmp)
    os.replace(tmp, LIB)
    return LIB


def _check_no_missing_kernels(lib):
    """Fail the build if any kernel launch stub is left undefined (a kernel
    the host pass silently did not instantiate)."""
    r = subprocess.run(["nm", "-D", "--undefined-only", lib], capture_output=True, text=True)
    if r.returncode != 0:
        return  # nm unavailable: the loader will report it instead
    missing = [l.split()[-1] for l in r.stdout.splitlines() if "__device_stub__" in l]
    if missing:
        raise RuntimeError(f"{len(missing)} kernel stubs undefined in {lib}, e.g. {missing[0]}")


if __name__ == "__main__":
    build(verbose="-q" not in sys.argv)

"""Build the gfx950 HIP library paper_2301_12457_amd/libevox.so in-tree.

Every translation unit is compiled by hipcc for gfx950 only, in parallel:
one per benchmark function (evox_fn.hip with -DEVOX_FN=<id>), the
function-independent kernels (evox_common.hip) and the C ABI
(evox_api.cpp), then linked into one shared library.

Flags: -ffp-contract=off (fused multiply-adds only where fmaf() is written,
so the elementwise updates are reproducible), and packed-fp32 instructions
disabled.
"""
import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OUT = os.path.join(HERE, "libevox.so")
BUILD_DIR = os.path.join(HERE, "_build")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
N_FN = 6

COMMON_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-ffp-contract=off",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function", f"-I{INCLUDE}", f"-I{CSRC}",
]


def _units():
    units = []
    for fn in range(N_FN):
        units.append((os.path.join(CSRC, "evox_fn.hip"), f"evox_fn{fn}.o", [f"-DEVOX_FN={fn}"]))
    units.append((os.path.join(CSRC, "evox_common.hip"), "evox_common.o", []))
    units.append((os.path.join(CSRC, "evox_gemm.hip"), "evox_gemm.o", []))
    units.append((os.path.join(CSRC, "evox_maes.hip"), "evox_maes.o", []))
    units.append((os.path.join(CSRC, "evox_nsga2.hip"), "evox_nsga2.o", []))
    units.append((os.path.join(CSRC, "evox_api.cpp"), "evox_api.o", ["-x", "hip"]))
    return units


def _compile(unit, verbose):
    src, obj, extra = unit
    out = os.path.join(BUILD_DIR, obj)
    cmd = [HIPCC] + COMMON_FLAGS + extra + ["-c", src, "-o", out]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    errs = "\n".join(l for l in r.stderr.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {os.path.basename(src)} {extra}:\n{errs}")
    if errs.strip() and verbose:
        print(errs, flush=True)
    return out


def build(verbose: bool = False, jobs: int = 8) -> str:
    os.makedirs(BUILD_DIR, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(lambda u: _compile(u, verbose), _units()))
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", OUT + ".tmp"] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(OUT + ".tmp", OUT)
    return OUT


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
    print(OUT)

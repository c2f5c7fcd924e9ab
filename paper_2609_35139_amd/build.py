"""Build the in-tree HIP C-ABI library ``libcacherepair.so`` for gfx950.

Every call recompiles all sources (hipcc cross-compiles without a GPU) and
atomically replaces the library next to this file.
"""
import concurrent.futures
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
SOURCES = ["api.hip", "gemm.hip", "attention.hip", "rowops.hip"]
# Per-source code generation options.  The attention kernel's score and
# output accumulators are read by VALU code every key tile; keeping MFMA
# operands in VGPRs avoids a copy out of the accumulation registers per tile.
EXTRA = {"attention.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"]}
LIB = os.path.join(HERE, "libcacherepair.so")
ARCH = "gfx950"
CFLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-fPIC", "-std=c++17",
    # packed fp32 VALU forms are kept out of every kernel
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"),
]


def _hipcc() -> str:
    return os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    return out


def build(verbose: bool = False) -> str:
    objdir = os.path.join(HERE, "_build")
    os.makedirs(objdir, exist_ok=True)
    jobs = []
    for src in SOURCES:
        obj = os.path.join(objdir, src.replace(".hip", ".o"))
        jobs.append(([_hipcc(), *CFLAGS, *EXTRA.get(src, []), "-c", os.path.join(CSRC, src),
                      "-o", obj], obj))
    workers = max(1, min(len(jobs), int(os.environ.get("MAX_JOBS", "4"))))
    with concurrent.futures.ThreadPoolExecutor(workers) as ex:
        for out in ex.map(_run, [j[0] for j in jobs]):
            if verbose and out.strip():
                print(out)
    tmp = LIB + ".tmp"
    _run([_hipcc(), f"--offload-arch={ARCH}", "-shared", "-o", tmp, *[j[1] for j in jobs],
          f"-Wl,--version-script={os.path.join(CSRC, 'exports.map')}"])
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))

"""Build the in-tree HIP C-ABI library ``libcacherepair.so`` for gfx950.

Every call recompiles all sources (hipcc cross-compiles without a GPU) and
atomically replaces the library next to this file.
"""
import concurrent.futures
import os
import re
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


RESOURCES = os.path.join(HERE, "_build", "kernel_resources.txt")


def _resources(remarks):
    """(kernel, VGPRs, scratch bytes per lane, waves per SIMD) from the
    compiler's kernel-resource-usage remarks."""
    rows, cur = [], None
    for line in remarks.splitlines():
        m = re.search(r"remark:\s+(Function Name|VGPRs|ScratchSize \[bytes/lane\]|"
                      r"Occupancy \[waves/SIMD\]):\s+(\S+)", line)
        if not m:
            continue
        key, val = m.group(1), m.group(2)
        if key == "Function Name":
            cur = {"kernel": val}
            rows.append(cur)
        elif cur is not None:
            cur[key.split()[0]] = int(val)
    return rows


def build(verbose: bool = False) -> str:
    objdir = os.path.join(HERE, "_build")
    os.makedirs(objdir, exist_ok=True)
    jobs = []
    for src in SOURCES:
        obj = os.path.join(objdir, src.replace(".hip", ".o"))
        jobs.append(([_hipcc(), *CFLAGS, *EXTRA.get(src, []), "-Rpass-analysis=kernel-resource-usage",
                      "-c", os.path.join(CSRC, src), "-o", obj], obj))
    workers = max(1, min(len(jobs), int(os.environ.get("MAX_JOBS", "4"))))
    rows = []
    with concurrent.futures.ThreadPoolExecutor(workers) as ex:
        for out in ex.map(_run, [j[0] for j in jobs]):
            rows += _resources(out)
            rest = "\n".join(l for l in out.splitlines() if "kernel-resource-usage" not in l)
            if verbose and rest.strip():
                print(rest)
    # per-kernel register and scratch use of the compiled kernels (a spill to scratch
    # memory in a hot kernel is a performance bug the tests look for)
    with open(RESOURCES, "w") as fh:
        for r in rows:
            fh.write("%s vgprs=%s scratch=%s waves=%s\n" % (
                r["kernel"], r.get("VGPRs"), r.get("ScratchSize"), r.get("Occupancy")))
    tmp = LIB + ".tmp"
    _run([_hipcc(), f"--offload-arch={ARCH}", "-shared", "-o", tmp, *[j[1] for j in jobs],
          f"-Wl,--version-script={os.path.join(CSRC, 'exports.map')}"])
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))

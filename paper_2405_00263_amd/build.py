"""Build libclover.so (HIP, gfx950) in-tree with hipcc.

Every call recompiles all sources; objects go to ``_build/`` next to this file and the
shared library to ``libclover.so`` in this directory.
"""
import os
import re
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libclover.so")
BUILD = os.path.join(HERE, "_build")
ARCH = "gfx950"
SOURCES = ["gemm.hip", "gemm_tiled.hip", "gemm_wide.hip", "gemm_wide_acc.hip", "attention.hip", "rows.hip", "tree.hip", "api.cpp", "noalloc.hip"]
# per-source extra flags: the 32x32 matrix-core kernel's 128-row shapes keep their accumulators
# in VGPRs (the alternative form moves them between register files inside the loop); its
# 256-row shape (gemm_wide_acc.hip) needs the accumulation registers and takes the default
EXTRA_FLAGS = {"gemm_wide.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form=1"]}
CFLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
          # per-kernel resource report, read by _check_no_scratch
          "-Rpass-analysis=kernel-resource-usage",
          # packed fp32 instructions stay off (see the project notes on gfx950 correctness)
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-Wno-unused-command-line-argument"]


def _hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc"):
        if c and os.path.exists(c):
            return c
    return "hipcc"


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if r.returncode != 0:
        raise RuntimeError("build failed:\n" + " ".join(cmd) + "\n" + r.stdout)
    return r.stdout


def _check_no_scratch(report: str, source: str):
    """Fail the build if a kernel uses private (scratch) memory: in these kernels that only
    happens when an accumulator array is indexed at run time, which moves it out of
    registers and slows the kernel several-fold."""
    name = None
    bad = []
    for line in report.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            name = m.group(1)
            continue
        m = re.search(r"ScratchSize \[bytes/lane\]: (\d+)", line)
        if m and int(m.group(1)) > 0:
            bad.append(f"{name}: {m.group(1)} bytes/lane")
    if bad:
        raise RuntimeError(f"{source}: kernels using scratch memory:\n  " + "\n  ".join(bad))


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    hipcc = _hipcc()
    objs, cmds = [], []
    for s in SOURCES:
        o = os.path.join(BUILD, os.path.splitext(s)[0] + ".o")
        objs.append(o)
        cmds.append([hipcc, *CFLAGS, *EXTRA_FLAGS.get(s, []), "-c", os.path.join(SRC, s), "-o", o])
    with ThreadPoolExecutor(max_workers=min(len(cmds), os.cpu_count() or 4)) as ex:
        for src, out in zip(SOURCES, ex.map(_run, cmds)):
            _check_no_scratch(out, src)
            if verbose:
                warn = "\n".join(l for l in out.splitlines() if "remark:" not in l)
                if warn.strip():
                    print(warn)
    tmp = OUT + ".tmp"
    _run([hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs])
    os.replace(tmp, OUT)
    if verbose:
        print("built", OUT)
    return OUT


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)

"""Build libsonic.so (the HIP kernels and the C ABI) for gfx950, in-tree.

    python -m paper_2601_21927_amd.build

Each .hip source is compiled to an object with hipcc, in parallel, then linked
into ``paper_2601_21927_amd/libsonic.so``.  Packed-FP32 instructions are
disabled for device code; the build then checks the generated gfx950
assembly of its own sources for them.
"""
from __future__ import annotations

import concurrent.futures
import glob
import os
import re
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libsonic.so")
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", shutil.which("hipcc") or "/opt/rocm/bin/hipcc")
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-variable",
    # M0 is declared clobbered by the direct-to-LDS inline assembly on purpose; the
    # build checks that no compiler-generated code uses it (_check_m0_only_in_asm)
    "-Wno-inline-asm",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]
PACKED_FP32 = re.compile(r"\bv_pk_(fma|mul|add)_f32\b")


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.basename(src).replace(".hip", ".o"))
    cmd = [HIPCC, *FLAGS, "-c", src, "-o", obj, "-save-temps=obj"]
    # keep the temporaries (device assembly) beside the object, inside _build/
    r = subprocess.run(cmd, cwd=BUILD, capture_output=True, text=True)
    noise = "'-packed-fp32-ops' is not a recognized feature for this target"
    err = "\n".join(l for l in r.stderr.splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{err}")
    if err.strip():
        sys.stderr.write(err + "\n")
    return obj


def _check_no_packed_fp32():
    bad = []
    for s in glob.glob(os.path.join(BUILD, "*-hip-amdgcn-amd-amdhsa-*.s")):
        with open(s) as f:
            for ln, line in enumerate(f, 1):
                if PACKED_FP32.search(line.split(";", 1)[0]):
                    bad.append(f"{os.path.basename(s)}:{ln}: {line.strip()}")
    if bad:
        raise RuntimeError("packed-FP32 instructions in device code:\n" + "\n".join(bad[:20]))


def _check_m0_only_in_asm():
    """The direct-to-LDS loads set M0 inside inline assembly that declares it
    clobbered; the compiler does not preserve a reserved register across such a
    statement, so no compiler-generated code may rely on M0 anywhere."""
    bad = []
    for s in glob.glob(os.path.join(BUILD, "*-hip-amdgcn-amd-amdhsa-*.s")):
        in_asm = False
        with open(s) as f:
            for ln, line in enumerate(f, 1):
                if ";;#ASMSTART" in line:
                    in_asm = True
                elif ";;#ASMEND" in line:
                    in_asm = False
                elif not in_asm and re.search(r"\bm0\b", line.split(";", 1)[0]):
                    bad.append(f"{os.path.basename(s)}:{ln}: {line.strip()}")
    if bad:
        raise RuntimeError("compiler-generated code uses M0:\n" + "\n".join(bad[:20]))


def build(verbose: bool = True) -> str:
    os.makedirs(BUILD, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(_compile, srcs))
    _check_no_packed_fp32()
    _check_m0_only_in_asm()
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stderr)
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


if __name__ == "__main__":
    build()

"""Build libdge.so (the HIP kernels + C ABI) in-tree for gfx950 with hipcc.

Usage: ``python -m paper_2609_33334_amd.build`` or ``build()`` from Python.
Objects go to ``_build/`` at the repository root; the shared library is written
next to this file so that it travels with the source tree.

Every source that issues global loads from inline asm (registers the compiler does not
track) is also compiled to gfx950 assembly and checked (``isa_check``): each such load is
waited on before its registers are touched on every path, and no kernel of the file
spills.  A violation raises ``BuildCheckError`` and no library is written.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys
import tempfile

from . import isa_check

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OBJDIR = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libdge.so")
ARCH = os.environ.get("DGE_OFFLOAD_ARCH", "gfx950")

HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
CFLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-result",
    f"-I{INCLUDE}", f"-I{CSRC}",
    # keep the compiler from forming packed fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


# Per-file additions.  score.hip, h2o.hip: MFMA accumulators in ordinary VGPRs, which saves the
# accumulator-to-VGPR copies before every softmax update (measured faster on MI355X), and
# no NaN semantics (inputs are finite; fmaxf then needs no canonicalising moves).
FILE_FLAGS = {
    "score.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form", "-fno-honor-nans"],
    "h2o.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form", "-fno-honor-nans"],
}


class BuildCheckError(RuntimeError):
    """The generated code of a source breaks a property its kernels rely on."""


def flags_for(src: str) -> list:
    return [*CFLAGS, *FILE_FLAGS.get(os.path.basename(src), [])]


def sources(csrc: str = CSRC):
    return sorted(os.path.join(csrc, f) for f in os.listdir(csrc) if f.endswith(".hip"))


def _compile(src: str, objdir: str, extra=()) -> str:
    obj = os.path.join(objdir, os.path.basename(src) + ".o")
    cmd = [HIPCC, *flags_for(src), *extra, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    return obj


def verify_source(src: str, extra=()) -> list:
    """Compile one source to gfx950 assembly (device code only, the library's flags plus
    ``extra``) and check its asm loads and private segments.  Returns the problems found
    (empty when the source issues no asm loads or passes)."""
    with open(src) as fh:
        if not isa_check.uses_asm_loads(fh.read()):
            return []
    flags = [f for f in flags_for(src) if f != "-fPIC"]
    with tempfile.TemporaryDirectory() as tmp:
        out = os.path.join(tmp, os.path.basename(src) + ".s")
        r = subprocess.run([HIPCC, *flags, *extra, "-S", "--cuda-device-only", src, "-o", out],
                           capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc -S failed for {src}:\n{r.stdout}\n{r.stderr}")
        report: list = []
        n, bad, spills = isa_check.check_asm(out, report=report)
    if n == 0:
        report.append(f"{os.path.basename(src)}: uses asm loads but none found in its "
                      "assembly (checker out of date?)")
    return [f"{os.path.basename(src)}: {p}" for p in report]


def build(verbose: bool = False, srcs=None, lib_path: str = LIB, objdir: str = OBJDIR,
          extra_flags=()) -> str:
    """Compile ``srcs`` (default: every .hip file of csrc/) and link ``lib_path``.
    Sources with asm loads are verified first; on a violation nothing is written."""
    os.makedirs(objdir, exist_ok=True)
    srcs = sources() if srcs is None else list(srcs)
    workers = max(1, min(8, os.cpu_count() or 1))
    with cf.ThreadPoolExecutor(workers) as ex:
        checks = [ex.submit(verify_source, s, extra_flags) for s in srcs]
        objs = [ex.submit(_compile, s, objdir, extra_flags) for s in srcs]
        problems = [p for c in checks for p in c.result()]
        objs = [o.result() for o in objs]
    if problems:
        raise BuildCheckError("generated code check failed, library not written:\n  "
                              + "\n  ".join(problems[:40]))
    tmp = lib_path + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, lib_path)
    if verbose:
        print(f"built {lib_path} (asm-load and spill checks passed)")
    return lib_path


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)

"""Generated-code checks that build() runs before it writes libdge.so (CPU only).

The scoring kernels issue register loads from inline asm that the compiler does not
track; build() compiles such sources to gfx950 assembly and refuses the library when a
load's registers are touched before a covering wait on some path, or when a kernel of
the file spills.  These tests run that check on every such source and show that build()
refuses a kernel forced to spill."""
import os
import tempfile

import pytest

from paper_2609_33334_amd import build, isa_check

# A kernel with asm register loads in the style of the scoring kernels.  SPILL_ATTR caps
# its registers so that the compiler has to spill.
_KERNEL = r"""
#include "dge_device.hpp"
using namespace dge;
__global__ SPILL_ATTR void probe_kernel(const uint4* src, float* out, int n) {
  u32x4_t v[12];
#pragma unroll
  for (int i = 0; i < 12; ++i) v[i] = async_load16(src + (size_t)i * n + threadIdx.x);
  asm_wait_vmcnt<0>();
#pragma unroll
  for (int i = 0; i < 12; ++i) reg_fence(v[i]);
  float acc = 0.0f;
#pragma unroll
  for (int i = 0; i < 12; ++i)
#pragma unroll
    for (int j = 0; j < 12; ++j)
      acc += __uint_as_float(v[i].x ^ v[j].y) * __uint_as_float(v[j].z | v[i].w);
  out[threadIdx.x] = acc;
}
"""


def _write(tmp, attr):
    src = os.path.join(tmp, "probe.hip")
    with open(src, "w") as fh:
        fh.write(_KERNEL.replace("SPILL_ATTR", attr))
    return src


ASM_LOAD_SOURCES = ("score.hip", "h2o.hip", "attend.hip", "project.hip")


@pytest.mark.parametrize("name", ASM_LOAD_SOURCES)
def test_asm_loads_waited_on_every_path(name):
    src = os.path.join(build.CSRC, name)
    with open(src) as fh:
        assert isa_check.uses_asm_loads(fh.read())
    problems = build.verify_source(src)
    assert problems == [], "\n".join(problems[:20])


def test_every_asm_load_source_is_listed():
    users = []
    for src in build.sources():
        with open(src) as fh:
            if isa_check.uses_asm_loads(fh.read()):
                users.append(os.path.basename(src))
    assert sorted(users) == sorted(ASM_LOAD_SOURCES)


def test_build_refuses_a_spilling_asm_load_kernel():
    with tempfile.TemporaryDirectory() as tmp:
        src = _write(tmp, "__attribute__((amdgpu_num_vgpr(24)))")
        lib = os.path.join(tmp, "libprobe.so")
        with pytest.raises(build.BuildCheckError, match="spills"):
            build.build(srcs=[src], lib_path=lib, objdir=tmp)
        assert not os.path.exists(lib)


def test_build_accepts_the_same_kernel_without_spills():
    with tempfile.TemporaryDirectory() as tmp:
        src = _write(tmp, "")
        lib = os.path.join(tmp, "libprobe.so")
        build.build(srcs=[src], lib_path=lib, objdir=tmp)
        assert os.path.exists(lib)


def test_checker_flags_a_read_before_the_wait():
    # hand-written assembly: the destination of an asm load is read with no wait between
    asm = "\n".join([
        "_Z1kv:",
        ";;#ASMSTART",
        "global_load_dwordx4 v[4:7], v[0:1], off",
        ";;#ASMEND",
        "v_add_f32 v8, v4, v5",
        "s_waitcnt vmcnt(0)",
        "s_endpgm",
        "_Z1jv:",
        ";;#ASMSTART",
        "global_load_dwordx4 v[4:7], v[0:1], off",
        ";;#ASMEND",
        "global_load_dword v9, v[2:3], off",
        "s_waitcnt vmcnt(1)",
        "v_add_f32 v8, v4, v5",
        "s_endpgm",
    ])
    with tempfile.TemporaryDirectory() as tmp:
        p = os.path.join(tmp, "k.s")
        with open(p, "w") as fh:
            fh.write(asm)
        report = []
        n, bad, spills = isa_check.check_asm(p, report=report)
    assert (n, bad, spills) == (2, 1, 0), report
    assert "_Z1kv" in report[0]

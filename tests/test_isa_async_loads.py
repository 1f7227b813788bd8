"""The scoring kernels' asm register loads are never read before their wait (CPU only:
compiles score.hip to gfx950 assembly with the library's own flags)."""
import os
import subprocess
import tempfile

import pytest

from isa_async_check import check_file

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_score_asm_loads_waited_on_every_path():
    from paper_2609_33334_amd import build
    src = os.path.join(build.CSRC, "score.hip")
    flags = [f for f in build.flags_for(src) if f != "-fPIC"]
    with tempfile.TemporaryDirectory() as tmp:
        out = os.path.join(tmp, "score.s")
        r = subprocess.run([build.HIPCC, *flags, "-S", "--cuda-device-only", src, "-o", out],
                           capture_output=True, text=True)
        if r.returncode != 0:
            pytest.fail(f"hipcc failed:\n{r.stderr[-2000:]}")
        n, bad = check_file(out)
    assert n > 0, "no asm register loads found (checker out of date?)"
    assert bad == 0, f"{bad} asm register loads are read before their wait"

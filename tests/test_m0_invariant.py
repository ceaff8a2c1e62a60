"""The direct-to-LDS loads set M0 in inline assembly and list it as clobbered;
the compiler reserves M0 and warns that such a clobber may not be honoured.
That is safe only while the compiled kernels use M0 for nothing else.  This
test compiles the kernel source to gfx950 assembly (CPU only, no GPU) and
checks that every M0 reference is one of those writes, each followed at once
by the direct-to-LDS load that consumes it."""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "paper_2607_12505_amd", "csrc", "nmspmm_kernels.hip")


def _hipcc():
    for c in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if c and os.path.exists(c):
            return c
    return None


@pytest.mark.skipif(_hipcc() is None, reason="hipcc not available")
def test_m0_is_written_only_for_direct_to_lds_loads(tmp_path):
    out = tmp_path / "kernels.s"
    cmd = [_hipcc(), "--offload-arch=gfx950", "-O3", "-std=c++17", "--cuda-device-only", "-S",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-I", os.path.join(ROOT, "include"),
           SRC, "-o", str(out)]
    subprocess.run(cmd, check=True, stdout=subprocess.DEVNULL, stderr=subprocess.DEVNULL, timeout=600)
    # instructions only: drop comments, directives and labels
    lines = []
    for raw in out.read_text().splitlines():
        s = raw.split(";")[0].strip()
        if s and not s.startswith(".") and not s.endswith(":"):
            lines.append(s)
    writes = 0
    for i, s in enumerate(lines):
        if not re.search(r"\bm0\b", s):
            continue
        assert re.fullmatch(r"s_mov_b32 m0, s\d+", s), f"M0 used outside the direct-to-LDS helpers: {s}"
        assert re.match(r"global_load_lds_dword(x4)?\b", lines[i + 1]), f"M0 write not followed by its load: {s}"
        writes += 1
    assert writes > 0

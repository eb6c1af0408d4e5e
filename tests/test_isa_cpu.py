"""Checks on the gfx950 assembly of the prefill kernels (CPU: hipcc cross-compiles).

The direct global->LDS loads of the prefill are inline assembly that set the M0
register (the LDS destination) right before each load.  The compiler does not track
that clobber of a reserved register, so the kernels are correct only while nothing
else in them keeps a value in M0 across those loads: every instruction that names
M0 must be one of the load sequences."""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


@pytest.mark.skipif(not os.path.exists(HIPCC) and shutil.which("hipcc") is None,
                    reason="needs hipcc")
def test_prefill_m0_only_in_lds_load_sequences(tmp_path):
    out = tmp_path / "prefill.s"
    cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang", "-target-feature",
           "-Xclang", "-packed-fp32-ops", "-I", os.path.join(ROOT, "include"),
           "-I", os.path.join(ROOT, "paper_2608_02947_amd", "csrc"), "-x", "hip",
           "--cuda-device-only", "-S", os.path.join(ROOT, "paper_2608_02947_amd", "csrc", "prefill.hip"),
           "-o", str(out)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [ln.split(";")[0].strip() for ln in out.read_text().splitlines()]
    lines = [ln for ln in lines if ln and not ln.startswith(".")]
    n_seq = 0
    for i, ln in enumerate(lines):
        if not re.search(r"\bm0\b", ln):
            continue
        # the only allowed form: s_mov_b32 m0, <sgpr>; s_nop 0; global_load_lds_dwordx4
        assert re.match(r"s_mov_b32\s+m0,\s*s\d+$", ln), f"m0 used outside a load sequence: {ln}"
        assert lines[i + 1].startswith("s_nop") and lines[i + 2].startswith("global_load_lds_dwordx4"), \
            lines[i:i + 3]
        n_seq += 1
    assert n_seq > 0

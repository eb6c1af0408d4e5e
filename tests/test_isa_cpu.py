"""Checks on the gfx950 assembly of the kernels (CPU: hipcc cross-compiles).

The direct global->LDS loads of the prefill are inline assembly that set the M0
register (the LDS destination) right before each load.  The compiler does not track
that clobber of a reserved register, so the kernels are correct only while nothing
else in them keeps a value in M0 across those loads: every instruction that names
M0 must be one of the load sequences.

The kernels skip the MFMAs of pruned chunks and pairs by wave-uniform branches.  An
MFMA placed under an EXEC mask instead (a branch the compiler took for divergent)
still accumulates when the mask is all zero, so no MFMA may follow an EXEC-mask
write without a branch or a label in between."""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


needs_hipcc = pytest.mark.skipif(not os.path.exists(HIPCC) and shutil.which("hipcc") is None,
                                 reason="needs hipcc")


def _assembly(tmp_path, src):
    out = tmp_path / (src + ".s")
    cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang", "-target-feature",
           "-Xclang", "-packed-fp32-ops", "-I", os.path.join(ROOT, "include"),
           "-I", os.path.join(ROOT, "paper_2608_02947_amd", "csrc"), "-x", "hip",
           "--cuda-device-only", "-S", os.path.join(ROOT, "paper_2608_02947_amd", "csrc", src),
           "-o", str(out)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    return out.read_text()


@needs_hipcc
def test_prefill_m0_only_in_lds_load_sequences(tmp_path):
    lines = [ln.split(";")[0].strip() for ln in _assembly(tmp_path, "prefill.hip").splitlines()]
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


def _mfmas_under_exec_mask(asm):
    """(kernel, line) of every MFMA whose nearest preceding control point is a write
    of EXEC other than its restore at a join (s_or_b64 exec, exec, ...)."""
    bad, n_mfma, kernel = [], 0, None
    last = None  # the last control point: "label", "branch", "restore" or "mask"
    for raw in asm.splitlines():
        ln = raw.split(";")[0].strip()
        if not ln:
            continue
        m = re.match(r"^(_Z\w+):$", ln)
        if m:
            kernel, last = m.group(1), "label"
            continue
        if ln.endswith(":"):
            last = "label"
        elif ln.startswith("s_cbranch") or ln.startswith("s_branch"):
            last = "branch"
        elif re.match(r"^s_or_b64\s+exec,\s*exec,", ln):
            last = "restore"
        elif re.match(r"^s_\w+_b64\s+exec,", ln) or re.match(r"^s_\w+_saveexec_b64\s", ln):
            last = "mask"
        elif ln.startswith("v_mfma"):
            n_mfma += 1
            if last == "mask":
                bad.append((kernel, ln))
    return bad, n_mfma


@needs_hipcc
@pytest.mark.parametrize("src", ["prefill.hip", "decode.hip"])
def test_no_mfma_under_exec_mask(tmp_path, src):
    bad, n_mfma = _mfmas_under_exec_mask(_assembly(tmp_path, src))
    assert n_mfma > 0
    assert not bad, bad[:5]


def test_scratch_loop_check_finds_a_spill_in_a_loop():
    asm = """_Zk:
\tscratch_store_dword off, v1, off
.LBB0_1:                                ; =>This Inner Loop Header: Depth=1
\tscratch_load_dword v1, off, off
.LBB0_2:
\tscratch_load_dword v2, off, off
.Lfunc_end0:
"""
    assert _scratch_in_loops(asm) == {"_Zk": [3, 1]}


def test_exec_mask_check_finds_a_masked_mfma():
    """The check itself: a masked MFMA is found, a branched-around one is not."""
    masked = """_Zk:
\ts_and_saveexec_b64 s[4:5], vcc
\tv_mfma_f32_32x32x16_bf16 v[0:15], v[16:19], v[20:23], v[0:15]
\ts_or_b64 exec, exec, s[4:5]
"""
    branched = """_Zk:
\ts_and_saveexec_b64 s[4:5], vcc
\ts_cbranch_execz .LBB0_2
\tv_mfma_f32_32x32x16_bf16 v[0:15], v[16:19], v[20:23], v[0:15]
.LBB0_2:
\ts_or_b64 exec, exec, s[4:5]
\tv_mfma_f32_32x32x16_bf16 v[0:15], v[16:19], v[20:23], v[0:15]
"""
    assert len(_mfmas_under_exec_mask(masked)[0]) == 1
    assert _mfmas_under_exec_mask(branched) == ([], 2)


def _scratch_in_loops(asm):
    """Per kernel of the assembly: (scratch instructions, those inside a loop).  A block
    is inside a loop when the compiler's block comment says so ("Loop Header" or "in
    Loop"); the kernel's straight-line prologue and epilogue are not."""
    out = {}
    name, in_loop = None, False
    for ln in asm.splitlines():
        m = re.match(r"^(_Z\S+):", ln)
        if m:
            name, in_loop = m.group(1), False
            out[name] = [0, 0]
            continue
        if name is None:
            continue
        if ln.startswith(".Lfunc_end"):
            name = None
            continue
        if re.match(r"^\.LBB\d+_\d+:", ln) or ln.startswith("; %bb."):
            in_loop = "Loop" in ln
        if re.match(r"\s+scratch_", ln):
            out[name][0] += 1
            out[name][1] += in_loop
    return out


@needs_hipcc
@pytest.mark.parametrize("src", ["prefill.hip", "decode.hip", "rotate.hip"])
def test_kernels_do_not_spill(tmp_path, src):
    """No kernel spills vector registers to scratch, and scalar spills (into vector
    register lanes, a v_writelane/v_readlane pair each) stay a handful: a mask or
    loop that keeps many lane masks live at once shows up here first.  The prefill
    kernels that rotate unrotated caches (third template argument true) hold the
    rotation's state beside the rest: they may spill up to 16 scalar registers (their
    reloads sit in the prologue and epilogue; the windowed d = 64 one adds two per
    tile) and up to 4 vector registers, provided that no scratch access lies inside a
    loop."""
    out = tmp_path / (src + ".o")
    cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang", "-target-feature",
           "-Xclang", "-packed-fp32-ops", "-I", os.path.join(ROOT, "include"),
           "-I", os.path.join(ROOT, "paper_2608_02947_amd", "csrc"), "-x", "hip",
           "--cuda-device-only", "-c", os.path.join(ROOT, "paper_2608_02947_amd", "csrc", src),
           "-o", str(out), "-Rpass-analysis=kernel-resource-usage"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    kernels = {}
    name = None
    for ln in r.stderr.splitlines():
        m = re.search(r"Function Name: (\S+)", ln)
        if m:
            name = m.group(1)
            kernels[name] = {}
            continue
        m = re.search(r"(VGPRs Spill|SGPRs Spill|ScratchSize \[bytes/lane\]): (\d+)", ln)
        if m and name:
            kernels[name][m.group(1)] = int(m.group(2))
    assert kernels
    loops = _scratch_in_loops(_assembly(tmp_path, src))
    for k, v in kernels.items():
        rotating = re.search(r"prefill_kernelILi\d+ELb[01]ELb1E", k) is not None
        if rotating:
            assert v.get("VGPRs Spill", 0) <= 4, (k, v)
            assert loops[k][1] == 0, (k, "scratch access inside a loop", loops[k])
        else:
            assert v.get("VGPRs Spill", 0) == 0 and v.get("ScratchSize [bytes/lane]", 0) == 0, \
                (k, v)
        assert v.get("SGPRs Spill", 0) <= (16 if rotating else 8), (k, v)

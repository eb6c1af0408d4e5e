"""The host code of libatf.so (window tables, closed-form counts, argument validation
of every entry point) and the C oracle under AddressSanitizer and
UndefinedBehaviorSanitizer, on the CPU.

Each builds a sanitized copy in a temporary directory (the host side only: the device
code of the HIP sources is compiled as usual) and runs the CPU tests that exercise it
in a child process with the sanitizer runtime preloaded: tests/test_abi_cpu.py for the
library (no device work), tests/test_oracle.py for the oracle.  A sanitizer report
fails the child (halt on error), and its output is checked for reports too."""
import glob
import importlib.util
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SAN_OPTS = {"ASAN_OPTIONS": "detect_leaks=0:halt_on_error=1:abort_on_error=0",
            "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"}


def _run_pytest(test_file, env_extra):
    env = dict(os.environ, OMP_NUM_THREADS="4", **SAN_OPTS, **env_extra)
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", test_file)],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-3000:]
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-3000:]
    return out


def test_oracle_under_asan_ubsan(tmp_path):
    so = tmp_path / "liboracle_san.so"
    subprocess.run(["gcc", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                    "-fno-sanitize-recover=undefined", "-fopenmp", "-fPIC", "-shared", "-std=c11",
                    "-o", str(so), os.path.join(ROOT, "oracle", "oracle.c"), "-lm"],
                   check=True, capture_output=True)
    asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True,
                          text=True, check=True).stdout.strip()
    _run_pytest("test_oracle.py", {"ORACLE_LIB": str(so), "LD_PRELOAD": asan})


def _clang_asan_runtime():
    libs = glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")
    return libs[0] if libs else None


@pytest.mark.skipif(not os.path.exists(HIPCC) or _clang_asan_runtime() is None,
                    reason="needs hipcc and the clang AddressSanitizer runtime")
def test_library_host_code_under_asan_ubsan(tmp_path):
    csrc = os.path.join(ROOT, "paper_2608_02947_amd", "csrc")
    flags = ["--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-sanitize-recover=undefined",
             "-Xarch_host", "-fno-omit-frame-pointer",
             "-I", os.path.join(ROOT, "include"), "-I", csrc]
    objs = []
    # the library's own source list (build.py), loaded without importing the package
    spec = importlib.util.spec_from_file_location(
        "atf_build_sources", os.path.join(ROOT, "paper_2608_02947_amd", "build.py"))
    build = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(build)
    for src in build.SOURCES:
        obj = str(tmp_path / (src.split(".")[0] + ".o"))
        subprocess.run([HIPCC, *flags, "-x", "hip", "-c", os.path.join(csrc, src), "-o", obj],
                       check=True, capture_output=True)
        objs.append(obj)
    lib = str(tmp_path / "libatf_san.so")
    subprocess.run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-shared-libsan",
                    "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                    "-o", lib, *objs], check=True, capture_output=True)
    _run_pytest("test_abi_cpu.py", {"ATF_LIB": lib, "LD_PRELOAD": _clang_asan_runtime()})

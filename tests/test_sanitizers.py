"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

* the oracle (oracle/mustafar_oracle.c) driven over random and edge-case inputs
  with exactly sized buffers (tests/sanitize/oracle_harness.c);
* the C ABI's host side (csrc/api.hip: validation, launch geometry, workspace
  layout, descriptor bookkeeping) with its kernel launchers replaced by stubs
  (tests/sanitize/launch_stubs.hip), every entry point called with valid,
  invalid and extreme arguments (tests/sanitize/abi_harness.c).

Only host code is instrumented: every hipcc line puts -Xarch_host before each
-fsanitize= flag (the device code is built as usual), and the link line adds
-fno-gpu-sanitize. The harnesses run on a machine without a GPU.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "tests", "sanitize")
CSRC = os.path.join(ROOT, "paper_2505_22913_amd", "csrc")
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
CLANG = "/opt/rocm/llvm/bin/clang"
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")

needs_toolchain = pytest.mark.skipif(not (os.path.exists(HIPCC) and os.path.exists(CLANG)),
                                     reason="ROCm clang / hipcc not installed")


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout[-3000:]}\n{r.stderr[-3000:]}"
    return r.stdout


@needs_toolchain
def test_oracle_is_clean_under_asan_and_ubsan(tmp_path):
    exe = str(tmp_path / "oracle_harness")
    _run([CLANG, "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
          "-fno-sanitize-recover=all", os.path.join(ROOT, "oracle", "mustafar_oracle.c"),
          os.path.join(SAN, "oracle_harness.c"), "-lm", "-o", exe])
    assert "oracle harness ok" in _run([exe], env=ENV)


@needs_toolchain
def test_abi_host_code_is_clean_under_asan_and_ubsan(tmp_path):
    host_san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                "-Xarch_host", "-fno-sanitize-recover=all"]
    common = ["--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fno-strict-aliasing",
              f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}"]
    api_o, stubs_o, main_o = (str(tmp_path / n) for n in ("api.o", "stubs.o", "harness.o"))
    _run([HIPCC, *common, *host_san, "-c", os.path.join(CSRC, "api.hip"), "-o", api_o])
    _run([HIPCC, *common, *host_san, "-c", os.path.join(SAN, "launch_stubs.hip"), "-o", stubs_o])
    _run([CLANG, "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
          f"-I{os.path.join(ROOT, 'include')}", "-c", os.path.join(SAN, "abi_harness.c"), "-o", main_o])
    exe = str(tmp_path / "abi_harness")
    _run([HIPCC, "-fsanitize=address,undefined", "-fno-gpu-sanitize", api_o, stubs_o, main_o, "-o", exe])
    assert "abi harness ok" in _run([exe], env=ENV)

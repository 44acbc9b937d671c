"""CPU builds with AddressSanitizer and UndefinedBehaviorSanitizer: the
oracle and the input generator (plain C, gcc) driven through their entry
points, and the C ABI's host code (hipcc, host side only; the kernel
launchers replaced by stand-ins) driven through every entry point on the
workloads' shapes, edge cases and argument errors.  A sanitizer report
fails the run."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
NATIVE = os.path.join(ROOT, "tests", "native")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1",
           UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")


def _run(cmd, **kw):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, **kw)
    assert r.returncode == 0, f"{' '.join(cmd[:3])} ... failed ({r.returncode}):\n{r.stdout[-4000:]}"
    return r.stdout


def test_oracle_and_generator_under_sanitizers(tmp_path):
    exe = str(tmp_path / "san_main")
    _run(["gcc", "-O1", "-g", "-std=c11", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
          "-fno-omit-frame-pointer", os.path.join(NATIVE, "sanitize_main.c"), os.path.join(ROOT, "oracle", "oracle.c"),
          os.path.join(ROOT, "datagen", "datagen.c"), "-o", exe, "-lm", "-pthread"])
    assert "ok" in _run([exe], env=ENV)


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc is not installed")
def test_abi_host_code_under_sanitizers(tmp_path):
    exe = str(tmp_path / "abi_san")
    csrc = os.path.join(ROOT, "paper_2010_05337_amd", "csrc")
    _run([HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17",
          "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
          "-Xarch_host", "-fno-sanitize-recover=all", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-I" + os.path.join(ROOT, "include"), "-I" + csrc, os.path.join(csrc, "api.hip"),
          os.path.join(NATIVE, "abi_stubs.cpp"), os.path.join(NATIVE, "abi_sanitize_main.cpp"), "-o", exe],
         cwd=str(tmp_path))
    # the HIP runtime's own allocations are not ours to audit: no leak check here
    env = dict(ENV, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1")
    assert "ok" in _run([exe], env=env, cwd=str(tmp_path))

"""Host sanitizer runs: the C oracle and the C-ABI layer's host code built
with AddressSanitizer and UndefinedBehaviorSanitizer into standalone
executables (every buffer they touch allocated by the instrumented runtime,
so an access past it is caught), driven over every function with ordinary,
empty and extreme arguments (tests/sanitize/).  Any sanitizer report aborts
the driver; a wrong status or result makes it exit nonzero.

The drivers are executables rather than the Python tests run under the
sanitizers: a sanitized library loaded into an uninstrumented interpreter
would see no redzones around numpy's buffers, and loading the runtime first
would need a preload of the interpreter itself."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
CSRC = os.path.join(ROOT, "paper_2608_02560_amd", "csrc")
INCLUDE = os.path.join(ROOT, "include")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SAN_HOST = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=all"]


def _run(cmd, cwd):
    res = subprocess.run(cmd, cwd=cwd, capture_output=True, text=True)
    assert res.returncode == 0, "%s\n%s\n%s" % (" ".join(cmd), res.stdout, res.stderr)
    return res


def _clean_env():
    env = dict(os.environ)
    env["ASAN_OPTIONS"] = "detect_leaks=1:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    return env


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_oracle_under_address_and_undefined_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_asan")
    _run(["gcc", "-O1", "-g", "-std=c11", "-fno-omit-frame-pointer", "-pthread",
          "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
          os.path.join(ROOT, "oracle", "precog_oracle.c"), os.path.join(HERE, "oracle_driver.c"),
          "-o", exe, "-lm"], str(tmp_path))
    res = subprocess.run([exe], capture_output=True, text=True, env=_clean_env(), timeout=300)
    assert res.returncode == 0, res.stdout + res.stderr
    assert "all checks passed" in res.stdout
    assert "runtime error" not in res.stderr and "AddressSanitizer" not in res.stderr


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="needs hipcc")
def test_abi_host_code_under_address_and_undefined_sanitizers(tmp_path):
    common = ["-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-I", INCLUDE, "-I", CSRC]
    host_only = ["-x", "hip", "--cuda-host-only"] + common + SAN_HOST
    objs = []
    for src in (os.path.join(CSRC, "precog_abi.cpp"), os.path.join(HERE, "launch_stubs.cpp"),
                os.path.join(HERE, "abi_driver.cpp")):
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        _run([HIPCC] + host_only + ["-c", src, "-o", obj], str(tmp_path))
        objs.append(obj)
    # the file with the library's device array keeps its device code; only
    # its host side is instrumented
    obj = str(tmp_path / "noalloc.hip.o")
    _run([HIPCC, "-x", "hip", "--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang",
          "-packed-fp32-ops"] + common + SAN_HOST +
         ["-c", os.path.join(CSRC, "noalloc.hip"), "-o", obj], str(tmp_path))
    objs.append(obj)
    exe = str(tmp_path / "abi_asan")
    _run([HIPCC, "--offload-arch=gfx950", "-Xarch_host", "-fsanitize=address", "-Xarch_host",
          "-fsanitize=undefined"] + objs + ["-o", exe], str(tmp_path))
    res = subprocess.run([exe], capture_output=True, text=True, env=_clean_env(), timeout=300)
    assert res.returncode == 0, res.stdout + res.stderr
    assert "all checks passed" in res.stdout
    assert "runtime error" not in res.stderr and "AddressSanitizer" not in res.stderr

"""Host sanitizer builds (CPU only): the C oracle and the C ABI's validation code run under
AddressSanitizer and UndefinedBehaviorSanitizer.

* The oracle is built with gcc and driven by tests/sanitize/oracle_driver.c, which calls every
  oracle function on small and degenerate shapes with buffers exactly as large as their shapes.
* The ABI's host code (api.cpp) is built with the sanitizers on its host pass only, linked with
  the library's other (unsanitized) objects, and driven by tests/sanitize/abi_driver.cpp, which
  calls every entry point with arguments that fail validation, so nothing reaches a GPU.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "tests", "sanitize")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
           UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")


def run(cmd, cwd, env=None, timeout=240):
    r = subprocess.run(cmd, cwd=cwd, env=env, capture_output=True, text=True, timeout=timeout)
    return r.returncode, r.stdout + r.stderr


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_oracle_under_address_and_undefined_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_asan")
    rc, out = run(["gcc", "-std=c11", "-O1", "-g", "-fsanitize=address,undefined",
                   "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
                   os.path.join(ROOT, "oracle", "dvref.c"), os.path.join(SAN, "oracle_driver.c"),
                   "-o", exe, "-lm"], str(tmp_path))
    assert rc == 0, out
    rc, out = run([exe], str(tmp_path), env=ENV)
    assert rc == 0 and out.strip().endswith("ok"), out


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")
def test_abi_validation_under_address_and_undefined_sanitizers(tmp_path):
    from paper_2609_34972_amd import build
    objs = [os.path.join(build.BUILD, os.path.splitext(s)[0] + ".o")
            for s in build.SOURCES if s != "api.cpp"]
    if not all(os.path.exists(o) for o in objs):
        build.build()
    host_san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                "-Xarch_host", "-fno-omit-frame-pointer"]
    api_o, drv_o, exe = (str(tmp_path / n) for n in ("api.o", "drv.o", "abi_asan"))
    rc, out = run([HIPCC, "-O1", "-g", "-std=c++17", "-fPIC", "--offload-arch=" + build.ARCH]
                  + host_san + ["-I", build.CSRC, "-c", os.path.join(build.CSRC, "api.cpp"),
                                "-o", api_o], str(tmp_path))
    assert rc == 0, out
    rc, out = run([HIPCC, "-O1", "-g", "-std=c++17"] + host_san
                  + ["-c", os.path.join(SAN, "abi_driver.cpp"), "-o", drv_o], str(tmp_path))
    assert rc == 0, out
    rc, out = run([HIPCC, "--offload-arch=" + build.ARCH] + host_san + [drv_o, api_o] + objs
                  + ["-o", exe], str(tmp_path))
    assert rc == 0, out
    # the HIP runtime keeps allocations of its own until exit; only memory errors are checked
    env = dict(ENV, ASAN_OPTIONS="detect_leaks=0")
    rc, out = run([exe], str(tmp_path), env=env)
    assert rc == 0 and out.strip().endswith("ok"), out

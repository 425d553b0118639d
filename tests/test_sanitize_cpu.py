"""CPU builds under AddressSanitizer and UndefinedBehaviorSanitizer:

* the oracle (oracle/pso.c) with a C driver that runs its whole pipeline on
  small seeded shapes (tests/sanitize/pso_driver.c);
* the library's host code -- the C ABI (csrc/psc_api.cpp) and the launch
  planners (csrc/conv_stream_launch.hip, csrc/conv_rows_launch.hip), compiled
  host-only with the sanitizers and linked with the library's other objects
  -- with a driver that makes every call that needs no GPU: library
  selection on edge values, configuration and workspace queries over a grid
  of shapes, and the argument checks of every entry point
  (tests/sanitize/abi_driver.cpp).

Each driver exits non-zero on the first sanitizer report or unexpected
status."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "tests", "sanitize")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=0",
           UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    return r.returncode, r.stdout + r.stderr


def test_oracle_under_sanitizers(tmp_path):
    if not shutil.which("gcc"):
        pytest.skip("gcc not available")
    exe = str(tmp_path / "pso_driver")
    rc, out = _run(["gcc", "-std=c99", "-O1", "-g", "-fno-omit-frame-pointer", "-Wno-unknown-pragmas",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                    os.path.join(ROOT, "oracle", "pso.c"), os.path.join(SAN, "pso_driver.c"), "-o", exe, "-lm"])
    assert rc == 0, out
    rc, out = _run([exe], env=dict(ENV, ASAN_OPTIONS="detect_leaks=1:halt_on_error=1"), timeout=300)
    assert rc == 0 and "pso driver ok" in out, out


# host-only sanitized translation units (no device code: no kernels in them)
HOST_ONLY = ["psc_api.cpp", "conv_stream_launch.hip", "conv_rows_launch.hip"]


def test_library_host_code_under_sanitizers(tmp_path):
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    from paper_2003_06513_amd import build as pbuild
    pbuild.build(incremental=True)            # the library's own objects, up to date
    csrc = pbuild.CSRC
    flags = ["-O1", "-g", "-fPIC", "-std=c++17", "-fno-omit-frame-pointer", "-I", os.path.join(ROOT, "include"),
             "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-sanitize-recover=all"]
    objs = []
    for src in [os.path.join(csrc, f) for f in HOST_ONLY] + [os.path.join(SAN, "abi_driver.cpp")]:
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        lang = ["-x", "hip"] if src.endswith(".cpp") else []
        rc, out = _run([HIPCC] + lang + ["--offload-host-only", "-c", src, "-o", obj] + flags)
        assert rc == 0, out
        objs.append(obj)
    srcs = sorted(f for f in os.listdir(csrc) if f.endswith((".hip", ".cpp")))
    objs += [os.path.join(pbuild.OUT_DIR, f + ".o") for f in srcs if f not in HOST_ONLY]
    exe = str(tmp_path / "abi_driver")
    rc, out = _run([HIPCC, "--offload-arch=" + pbuild.ARCH] + objs +
                   ["-o", exe, "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined"])
    assert rc == 0, out
    rc, out = _run([exe], env=ENV, timeout=300)
    assert rc == 0 and "abi driver ok" in out, out

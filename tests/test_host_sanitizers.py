"""The host side of the library (plan building: grid, quadrature, neighbour
search, basis evaluation; the packed, sweep, spectral and stencil layouts;
the C ABI's argument validation and host-only entry export) built with
AddressSanitizer and UndefinedBehaviorSanitizer and driven over many grid,
basis, quadrature and sampling configurations by tests/host_sanitize.cpp.
No GPU: the kernel launchers are stand-ins that are never reached."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(ROOT, "paper_2209_13603_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")
def test_host_code_is_clean_under_asan_and_ubsan(tmp_path):
    exe = str(tmp_path / "host_sanitize")
    # each -fsanitize= applies to the host compilation only (-Xarch_host)
    san = []
    for f in ("-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=undefined",
              "-fno-omit-frame-pointer"):
        san += ["-Xarch_host", f]
    srcs = [os.path.join(HERE, "host_sanitize.cpp"), os.path.join(HERE, "host_sanitize_stubs.cpp")] + \
        [os.path.join(CSRC, f) for f in ("disco_plan.cpp", "disco_pack.cpp", "disco_spectral_plan.cpp",
                                         "disco_abi.cpp")]
    cmd = [HIPCC, "-O1", "-g", "-std=c++17", *san, "-I", os.path.join(ROOT, "include"), "-I", CSRC, *srcs,
           "-L/opt/rocm/lib", "-lrocprofiler-sdk-roctx", "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stdout + r.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=600, env=env)
    print(r.stdout[-2000:])
    assert r.returncode == 0, r.stdout[-4000:] + r.stderr[-4000:]
    assert "OK (0 failures)" in r.stdout

"""The C ABI's host code under AddressSanitizer and UndefinedBehaviorSanitizer
(no GPU): every library source is rebuilt with the sanitizers on the host
side only (-Xarch_host; the gfx950 device code is compiled as usual and never
launched) and linked with tests/sanitize/abi_validation.cpp, which drives the
argument validation of every entry point, the status strings, the
thread-local message and the size helpers with degenerate and very large
arguments.  Any sanitizer report or wrong status fails the test."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_26650_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer"]

pytestmark = pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")


def _build(tmp):
    sys.path.insert(0, os.path.join(ROOT, "paper_2606_26650_amd"))
    import build as lib_build          # the library's own source list and flags
    sys.path.pop(0)
    import concurrent.futures as cf
    flags = [f for f in lib_build.FLAGS]

    def compile_one(src):
        obj = os.path.join(tmp, os.path.splitext(src)[0] + ".o")
        cmd = [HIPCC, *flags, *lib_build.EXTRA.get(src, []), *SAN, "-g", "-c",
               os.path.join(CSRC, src), "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-3000:]
        return obj

    with cf.ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        objs = list(ex.map(compile_one, lib_build.SOURCES))
    drv = os.path.join(tmp, "abi_validation.o")
    cmd = [HIPCC, "-O1", "-g", "-std=c++17", "--offload-arch=gfx950", *SAN,
           "-I", os.path.join(ROOT, "include"), "-c",
           os.path.join(ROOT, "tests", "sanitize", "abi_validation.cpp"), "-o", drv]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    exe = os.path.join(tmp, "abi_validation")
    r = subprocess.run([HIPCC, "--offload-arch=gfx950", *SAN, drv, *objs, "-o", exe],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    return exe


@pytest.mark.slow
def test_abi_validation_under_asan_ubsan(tmp_path):
    exe = _build(str(tmp_path))
    env = dict(os.environ)
    # the HIP runtime keeps process-lifetime allocations: leaks are not ours
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=0:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    env["HIP_VISIBLE_DEVICES"] = ""
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env)
    out = r.stdout + r.stderr
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert "ok: 0 failure(s)" in r.stdout

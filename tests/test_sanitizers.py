"""The coordinator's host code under ThreadSanitizer and AddressSanitizer, on the simulated
device (no GPU): tests/native/coord_stress.cpp drives init, task creation, concurrent submits
from four threads, polling, statistics and launch-log readers, drain, shutdown and the failure
path (an injected launch failure).  coord.cpp, ops.cpp and plan.cpp are rebuilt with the host
sanitizer (device code is built as usual) and linked with the library's kernel objects from
the in-tree build.  A sanitizer report or a wrong completion count fails the test."""
import glob
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2307_04339_amd", "csrc")
BUILD = os.path.join(ROOT, "_build")
SAN_DIR = os.path.join(BUILD, "sanitize")
HOST_SRCS = ["coord.cpp", "ops.cpp", "plan.cpp"]
DRIVER = os.path.join(ROOT, "tests", "native", "coord_stress.cpp")


def _kernel_objs():
    return sorted(glob.glob(os.path.join(BUILD, "kern_*.hip.o")))


def _build(kind):
    """Build the stress driver with -fsanitize=<kind> on the host side; returns its path."""
    out = os.path.join(SAN_DIR, kind)
    os.makedirs(out, exist_ok=True)
    exe = os.path.join(out, "coord_stress")
    srcs = [os.path.join(CSRC, s) for s in HOST_SRCS] + [DRIVER]
    deps = srcs + glob.glob(os.path.join(CSRC, "*.h")) + [os.path.join(ROOT, "include", "miriam.h")] + _kernel_objs()
    if os.path.exists(exe) and os.path.getmtime(exe) >= max(os.path.getmtime(p) for p in deps):
        return exe
    flags = ["--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-I", os.path.join(ROOT, "include"), "-Xarch_host", f"-fsanitize={kind}"]
    procs, objs = [], []
    for s in srcs:
        o = os.path.join(out, os.path.basename(s) + ".o")
        objs.append(o)
        procs.append(subprocess.Popen(["hipcc", "-x", "hip"] + flags + ["-c", s, "-o", o],
                                      stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True))
    for p in procs:
        msg = p.communicate()[0]
        assert p.returncode == 0, msg
    r = subprocess.run(["hipcc", "--offload-arch=gfx950", "-Xarch_host", f"-fsanitize={kind}", "-o", exe]
                       + objs + _kernel_objs() + ["-lpthread"], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    return exe


@pytest.mark.skipif(shutil.which("hipcc") is None, reason="needs hipcc")
@pytest.mark.skipif(not _kernel_objs(), reason="needs the in-tree kernel objects (run the build first)")
@pytest.mark.parametrize("kind", ["thread", "address"])
def test_coordinator_clean_under_sanitizer(kind):
    exe = _build(kind)
    env = dict(os.environ)
    env["TSAN_OPTIONS"] = "halt_on_error=1 exitcode=66"
    env["ASAN_OPTIONS"] = "halt_on_error=1 exitcode=66 detect_leaks=1"
    r = subprocess.run([exe], capture_output=True, text=True, timeout=600, env=env)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "OK" in r.stdout
    assert "Sanitizer" not in out, out[-4000:]

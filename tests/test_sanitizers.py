"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only):
the threshold controller (controller.cpp) and the host side of libdlm
(configuration checks, workspace and cache layouts, the step planner, the
validation of every step entry point), each driven over random and
edge-case arguments by a driver in tests/sanitize/. GPU code is not
sanitized: the hipcc lines instrument the host pass only."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "paper_2606_29094_amd", "csrc")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=0", UBSAN_OPTIONS="print_stacktrace=1")

pytestmark = pytest.mark.slow


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, (" ".join(cmd), r.stdout[-3000:], r.stderr[-3000:])
    return r.stdout


def test_controller_under_sanitizers(tmp_path):
    exe = str(tmp_path / "ctl")
    _run(["g++", "-std=c++17", "-O1", "-g", *SAN, "-o", exe, os.path.join(SRC, "controller.cpp"),
          os.path.join(ROOT, "tests", "sanitize", "controller_driver.cpp")])
    out = _run([exe], env=ENV)
    assert "0 failures" in out


@pytest.mark.skipif(not os.path.exists("/opt/rocm/bin/hipcc"), reason="hipcc not installed")
def test_library_host_code_under_sanitizers(tmp_path):
    objs = []
    procs = []
    for f in ("runtime", "gemm", "gemm_dl", "rowwise", "attention", "ceiling"):
        o = str(tmp_path / f"{f}.o")
        objs.append(o)
        # each sanitizer flag applies to the host pass only
        cmd = ["/opt/rocm/bin/hipcc", "--offload-arch=gfx950", "-O1", "-g", "-fPIC", "-std=c++17",
               "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
               "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
               "-Xarch_host", "-fno-sanitize-recover=all",
               "-I", SRC, "-c", os.path.join(SRC, f + ".hip"), "-o", o]
        procs.append((cmd, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.PIPE,
                                            text=True)))
    for cmd, p in procs:
        out, err = p.communicate()
        assert p.returncode == 0, (" ".join(cmd), err[-3000:])
    drv = str(tmp_path / "driver.o")
    _run(["g++", "-std=c++17", "-O1", "-g", *SAN, "-c",
          os.path.join(ROOT, "tests", "sanitize", "planner_driver.cpp"), "-o", drv])
    exe = str(tmp_path / "planner")
    _run(["g++", *SAN, "-o", exe, *objs, drv, "-L/opt/rocm/lib", "-lamdhip64",
          "-Wl,-rpath,/opt/rocm/lib"])
    out = _run([exe], env=ENV)
    assert "0 failures" in out

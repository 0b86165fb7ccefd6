"""The library's host logic under the host address and undefined-behaviour
sanitizers (CPU only).

tests/sanitize/driver.cpp exercises everything that runs without a context:
workspace plans and job layouts for thousands of random and malformed
specs, the tick schedule, the planner, the delay fit, the interval of
Eq. 5, and the argument checks of every entry point.  It is linked with the
library's host sources (api.cpp, schedule.cpp, planner.cpp, and lin.hip for
the product's grid size) and with stand-ins for the kernel launches, built
by hipcc with the sanitizers on the host side only (GPU code is built as
usual and never runs).  Leak checking is off: the HIP runtime's own
start-up allocations live until exit.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2510_12494_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


@pytest.mark.timeout(900)
def test_host_logic_under_sanitizers(tmp_path):
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    exe = str(tmp_path / "host_checks")
    srcs = [os.path.join(CSRC, f) for f in ("api.cpp", "schedule.cpp", "planner.cpp", "lin.hip")]
    srcs += [os.path.join(ROOT, "tests", "sanitize", f) for f in ("stubs.cpp", "driver.cpp")]
    san = []
    for opt in ("-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=all",
                "-fno-omit-frame-pointer"):
        san += ["-Xarch_host", opt]
    cmd = [HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-Wno-pass-failed",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", *san, *srcs, "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True, cwd=str(tmp_path))
    noise = "is not a recognized feature for this target"
    msgs = "\n".join(l for l in (r.stdout + r.stderr).splitlines() if noise not in l)
    assert r.returncode == 0, msgs
    env = dict(os.environ)
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    env["HIP_VISIBLE_DEVICES"] = ""          # never a GPU, even where there is one
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "host checks passed" in r.stdout, out[-4000:]
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-4000:]

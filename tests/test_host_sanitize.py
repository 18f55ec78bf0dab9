"""The host side of the library under AddressSanitizer and
UndefinedBehaviorSanitizer (no GPU): the plan builder (`csrc/plan.hip`,
compiled for the host only) linked into a seeded fuzz driver
(`tests/host/plan_fuzz.cpp`) that feeds zigzag_partition and plan creation
valid and malformed problems and runs every host query of each plan.  A
sanitizer report aborts the driver; a wrong accept / reject verdict fails
it."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")
def test_plan_builder_under_sanitizers(tmp_path):
    exe = str(tmp_path / "plan_fuzz")
    cmd = [HIPCC, "--offload-host-only", "-O1", "-g", "-std=c++17",
           f"-I{os.path.join(ROOT, 'include')}", f"-I{os.path.join(ROOT, 'paper_2609_07108_amd', 'csrc')}",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all",
           "-x", "hip", os.path.join(ROOT, "paper_2609_07108_amd", "csrc", "plan.hip"),
           "-x", "c++", os.path.join(ROOT, "tests", "host", "plan_fuzz.cpp"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stdout + r.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe, "20000"], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-4000:]
    assert " 0 failures" in r.stdout, r.stdout

"""The HDP planners (libbs_hdp's C ABI) under the address and undefined-behaviour sanitizers.

tests/native/hdp_sanitized.cpp calls bs_hdp_offload_ratio and bs_hdp_plan on 2,000 seeded
random batches (1-300 sequences of up to four times the rank capacity, 1-64 ranks, all three
algorithms, random cost models, delta and bucket counts) and on their error paths, and checks
each plan's structure: every sequence placed exactly once, valid ranks, packed micro-batches
within capacity, outputs untouched by every failed call.  It is built here from the planner's
source with -fsanitize=address,undefined (host code only; the planners never touch the GPU), so
any out-of-bounds access, leak or undefined operation aborts the run."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("g++") is None, reason="no host C++ compiler")
def test_hdp_planners_clean_under_sanitizers(tmp_path):
    exe = str(tmp_path / "hdp_sanitized")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-ffp-contract=off",
           os.path.join(ROOT, "paper_2502_21231_amd", "csrc", "hdp.cpp"),
           os.path.join(ROOT, "tests", "native", "hdp_sanitized.cpp"), "-o", exe]
    subprocess.run(cmd, check=True, capture_output=True, timeout=300)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-4000:]
    assert r.stdout.startswith("ok "), r.stdout
    assert int(r.stdout.split()[1]) > 1000  # most batches are feasible

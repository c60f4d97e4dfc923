"""libbs_attn's host-side argument checks under the address and undefined-behaviour sanitizers.

capi.hip (the C ABI: validation, workspace layout, error messages, the allocation-free entry
point's checks) is compiled again with host-only instrumentation (-fno-gpu-sanitize: the device
code is not instrumented) and linked with the library's other objects into
tests/native/capi_sanitized.cpp, which makes only calls that fail validation before any device
work, so it needs no GPU.  Any out-of-bounds access, leak or undefined operation on those paths
aborts the run."""
import glob
import os
import subprocess

import pytest

from paper_2502_21231_amd import build as BLD

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
OTHERS = [os.path.splitext(s)[0] for s in BLD.SOURCES if s != "capi.hip"]


def test_capi_argument_checks_clean_under_sanitizers(tmp_path):
    objs = [os.path.join(BLD.BUILD, n + ".o") for n in OTHERS]
    if not all(os.path.exists(o) for o in objs):
        pytest.fail("the library's objects are not built (run __graft_entry__.build())")
    cc = BLD.hipcc()
    san = ["-fsanitize=address", "-fsanitize=undefined", "-fno-gpu-sanitize"]
    obj = str(tmp_path / "capi_sanitized.o")
    exe = str(tmp_path / "capi_sanitized")
    subprocess.run([cc, f"--offload-arch={BLD.ARCH}", "-O1", "-g", "-std=c++17", "-fPIC", *san,
                    "-fno-sanitize-recover=undefined", "-Xclang", "-target-feature", "-Xclang",
                    "-packed-fp32-ops", "-Wno-unused-result", "-Wno-unused-value", "-c",
                    os.path.join(BLD.CSRC, "capi.hip"), "-o", obj],
                   check=True, capture_output=True, timeout=600)
    subprocess.run([cc, f"--offload-arch={BLD.ARCH}", "-g", "-std=c++17", *san, obj, *objs,
                    os.path.join(ROOT, "tests", "native", "capi_sanitized.cpp"), "-o", exe],
                   check=True, capture_output=True, timeout=600)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-4000:]
    assert r.stdout.strip() == "ok", r.stdout

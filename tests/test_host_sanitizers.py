"""The host planner, host interpreter, scheduler and pipeline model under
AddressSanitizer and UndefinedBehaviorSanitizer: a fuzz driver over random
tensors, meshes, specs, flags and tunings, with every plan run through the
host interpreter on buffers of exactly the shard sizes.  Host code only
(g++; no GPU code is built or run).  CPU only."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2211_05322_amd", "csrc")
HOST_SOURCES = ["planner.cpp", "capi.cpp", "schedule.cpp", "pipeline.cpp"]


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_host_code_under_asan_ubsan(tmp_path):
    exe = tmp_path / "host_fuzz"
    san = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer"]
    cmd = ["g++", "-std=c++17", "-O1", "-g", *san, "-I", os.path.join(ROOT, "include"),
           *[os.path.join(CSRC, f) for f in HOST_SOURCES], os.path.join(ROOT, "tests", "c", "host_fuzz.cpp"),
           "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([str(exe), "150"], capture_output=True, text=True, timeout=600, env=env)
    assert r.returncode == 0 and r.stdout.startswith("ok"), (r.stdout + r.stderr)[-4000:]

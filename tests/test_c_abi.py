"""The boundary is a C ABI: a C99 program built against include/reshard.h
alone links libreshard.so and runs host-only calls (plan, queries, the host
interpreter, error paths).  CPU only."""

import ast
import os
import shutil
import subprocess
import sys

import pytest

from paper_2211_05322_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_c99_client_against_header(tmp_path):
    lib = B.load()._name
    exe = tmp_path / "abi_smoke"
    cmd = ["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic", "-D_ISOC11_SOURCE",
           "-I", os.path.join(ROOT, "include"), os.path.join(ROOT, "tests", "c", "abi_smoke.c"),
           lib, f"-Wl,-rpath,{os.path.dirname(lib)}", "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout + r.stderr


def test_binding_maps_one_hip_runtime():
    """A script that loads the library through the binding before importing
    torch itself still has exactly one HIP runtime mapped: the one torch's
    tensors and streams come from."""
    code = ("from paper_2211_05322_amd import binding as B; B.load(); import torch; "
            "print(sorted({l.split()[-1] for l in open('/proc/self/maps') if 'libamdhip64' in l}))")
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert r.returncode == 0, r.stderr
    maps = ast.literal_eval(r.stdout.strip().splitlines()[-1])
    assert len(maps) == 1, maps

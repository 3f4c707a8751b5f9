"""The host sources under AddressSanitizer and UndefinedBehaviorSanitizer.

plan.cpp, view.cpp and api.cpp (planners, rank views and tile maps, the
device entry points' validation and parameter building) are compiled with
g++ and -fsanitize=address,undefined together with tests/sanitize/
host_driver.cpp, which stubs the HIP calls and the kernel launchers (the
stubs check every table pointer a launcher receives against the bound
blob) and drives the C ABI over random contexts and the five workloads at
full size. Any sanitizer report, leak or failed check fails the test.
"""
import os
import shutil
import subprocess

import numpy as np
import pytest

from oracle import planner as P
from paper_2606_08476_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HOST = os.path.join(ROOT, "paper_2606_08476_amd", "csrc", "host")


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_host_sources_under_sanitizers(tmp_path):
    exe = tmp_path / "host_driver"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", "-I", os.path.join(ROOT, "include"),
           os.path.join(HOST, "plan.cpp"), os.path.join(HOST, "view.cpp"),
           os.path.join(HOST, "api.cpp"), os.path.join(ROOT, "tests", "sanitize", "host_driver.cpp"),
           "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    # the five workloads: name, CP degree, plan, rank rule, heads, lengths
    lines = []
    for name, w in synth.WORKLOADS.items():
        cu = synth.cu_seqlens(synth.doc_lengths(name))
        lines.append(" ".join(map(str, [name, w.cp, w.plan, w.rank, len(cu) - 1, w.hq, w.hkv, w.d,
                                        *cu.tolist()])))
    wl = tmp_path / "workloads.txt"
    wl.write_text("\n".join(lines) + "\n")
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([str(exe), str(wl)], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-6000:])
    assert "all checks passed" in r.stdout
    for name in synth.WORKLOADS:
        assert f"workload {name}:" in r.stdout

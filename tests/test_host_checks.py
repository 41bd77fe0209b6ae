"""Host code built with the address and undefined-behaviour sanitizers (CPU).

* The library's host-side planning (paper_2505_18629_amd/csrc/rv_plan.h:
  workspace capacities, prefill chunks, attention key splits), checked at
  the shapes of every benchmark workload (the 70B prefill of 8 x 8192
  tokens included) and at edge cases by tests/host/plan_check.cpp.
* The oracle's weight generator (oracle/weights.c), driven over the tensor
  and element indices the workloads reach; its values must equal those of
  the normally built library.
"""
import ctypes
import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]

pytestmark = pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")


def _build_and_run(tmp_path, compiler, sources, extra, name):
    exe = str(tmp_path / name)
    subprocess.run([compiler] + SAN + extra + sources + ["-o", exe, "-lm"], check=True, capture_output=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    return subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)


def test_planning_stays_in_bounds(tmp_path):
    r = _build_and_run(tmp_path, "g++", [os.path.join(ROOT, "tests", "host", "plan_check.cpp")],
                       ["-std=c++17", "-I", os.path.join(ROOT, "paper_2505_18629_amd", "csrc")], "plan_check")
    assert r.returncode == 0, r.stdout + r.stderr
    assert "all plans in bounds" in r.stdout
    assert "70b prefill B=8: 32 chunks" in r.stdout


def test_weight_generator_under_sanitizers(tmp_path):
    r = _build_and_run(tmp_path, "gcc", [os.path.join(ROOT, "tests", "host", "weights_check.c"),
                                         os.path.join(ROOT, "oracle", "weights.c")], ["-std=c11", "-fopenmp"],
                       "weights_check")
    assert r.returncode == 0, r.stdout + r.stderr
    lines = r.stdout.split("\n")
    assert lines[0].split()[1:] == [str(x) for x in oracle.splitmix64_stream(0, 4)]
    shape = type("S", (), {"dtype": "bf16", "init_std": 0.02})
    shape32 = type("S", (), {"dtype": "f32", "init_std": 0.02})
    for line in lines:
        if line.startswith("fill"):
            _, t, start, bf16, *vals = line.split()
            ref = oracle.fill(shape if int(bf16) else shape32, 7, int(t), int(start), 16)
            np.testing.assert_array_equal(np.array(vals, dtype=np.float64), ref)
        if line.startswith("bits"):
            idx = np.array([0, 5, 128256 * 8192 - 1], dtype=np.uint64)
            ref = oracle._load()
            got = [int(x) for x in line.split()[1:]]
            out = np.empty(3, dtype=np.uint32)
            ref.orc_bits_at(7, 561, idx.ctypes.data_as(ctypes.c_void_p), 3, 1, 0.02,
                            out.ctypes.data_as(ctypes.c_void_p))
            assert got == out.tolist()

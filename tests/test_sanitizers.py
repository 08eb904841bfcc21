"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

Builds the oracle (oracle/rvo.c) and librv's host-only planning code
(paper_2609_23286_amd/csrc/rv_plan.cpp) with gcc/g++ and
-fsanitize=address,undefined, each with a driver under tests/native/ that exercises
every function over many shapes, devices and edge cases (empty query subsets, budget 0
and N, empty memories, forced work plans).  Any invalid memory access or undefined
behaviour aborts the driver, which fails the test."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
NATIVE = os.path.join(ROOT, "tests", "native")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]


def build_and_run(cmd, exe, expect):
    subprocess.run(cmd, check=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1", OMP_NUM_THREADS="4")
    for k in ("RV_ATTN_SPLIT", "RV_ATTN_FIRST_PCT", "RV_ATTN_WG_PER_CU", "RV_ATTN_MIN_CHUNK",
              "RV_ATTN_SPLIT_SLACK"):
        env.pop(k, None)
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert expect in r.stdout


def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_check")
    build_and_run(["gcc", "-std=c11", "-fopenmp", *SAN, "-o", exe, os.path.join(NATIVE, "oracle_check.c"),
                   os.path.join(ROOT, "oracle", "rvo.c"), "-lm"], exe, "oracle OK")


def test_host_planning_under_sanitizers(tmp_path):
    exe = str(tmp_path / "host_logic_check")
    build_and_run(["g++", "-std=c++17", *SAN, "-o", exe, os.path.join(NATIVE, "host_logic_check.cpp"),
                   os.path.join(ROOT, "paper_2609_23286_amd", "csrc", "rv_plan.cpp")], exe, "host logic OK")

"""The resident schedule's tile division (paper_1511_00175_amd/csrc/
fc_partition.h: plain host arithmetic used when a plan is made and by
fc_plan_balance), checked on the CPU under AddressSanitizer and
UndefinedBehaviorSanitizer over thousands of random plans: every table
covers each tile once, round by round, and no block exceeds its LDS cap."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "c", "partition_check.cpp")
CSRC = os.path.join(ROOT, "paper_1511_00175_amd", "csrc")


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_partition_tables_are_valid(tmp_path):
    exe = tmp_path / "partition_check"
    build = ["g++", "-std=c++17", "-O1", "-g", "-Wall", "-Wextra", "-Werror", "-fsanitize=address,undefined",
             "-fno-sanitize-recover=all", f"-I{CSRC}", SRC, "-o", str(exe)]
    r = subprocess.run(build, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    # the environment is passed on unchanged; ASan is told not to insist on
    # coming first among the loaded libraries
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "all tables valid" in r.stdout

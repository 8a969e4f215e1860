"""The host planner and validators (paper_2608_11152_amd/csrc/plan.cpp) built with g++ under the address
and undefined-behaviour sanitizers and driven by randomized plans (tests/host_plan_check.cpp): coverage
of every page / query row / key range, partial-slot bookkeeping, determinism and the error codes, with
any sanitizer report failing the run.  CPU only; no HIP code is built here."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


@pytest.fixture(scope="module")
def checker(tmp_path_factory):
    cxx = shutil.which("g++")
    if cxx is None:
        pytest.skip("g++ is not available")
    exe = str(tmp_path_factory.mktemp("sanitized") / "host_plan_check")
    cmd = [cxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", f"-I{os.path.join(ROOT, 'include')}",
           os.path.join(HERE, "host_plan_check.cpp"), os.path.join(ROOT, "paper_2608_11152_amd", "csrc", "plan.cpp"),
           "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    return exe


def _run(exe, *args):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    return subprocess.run([exe, *args], capture_output=True, text=True, timeout=300, env=env)


@pytest.mark.parametrize("seed", ["1", "2", "3"])
def test_randomized_plans_under_sanitizers(checker, seed):
    r = _run(checker, "400", seed)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "ok:" in r.stdout and "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr


def test_checker_rejects_planted_mistakes(checker):
    r = _run(checker, "self-test")
    assert r.returncode == 0, r.stdout + r.stderr
    assert "planted mistakes rejected" in r.stdout

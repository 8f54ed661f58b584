"""AddressSanitizer and UndefinedBehaviorSanitizer builds of the host code (no GPU):
the prefix cache (csrc/kvx_cache.cpp) under random turn sequences of both
policies with host tiers, recency tiers and shared-prefix groups; the radix
tree (csrc/kvx_radix.cpp) under random branching request sequences; the work
planners of csrc/kvx_host.cpp under random ragged batches (kernel launchers
stubbed out); and the C oracle under random ragged batches stored into
NaN-filled pools.  The drivers also check ownership, coverage and finiteness
invariants; see tests/sanitize/."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]


def _build_and_run(cmd, exe, args, tmp_path):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        if "asan" in r.stderr.lower() or "ubsan" in r.stderr.lower():
            pytest.skip("sanitizer runtime not available: " + r.stderr[-300:])
        raise AssertionError(r.stderr[-3000:])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    run = subprocess.run([exe, *args], capture_output=True, text=True, env=env, timeout=600, cwd=tmp_path)
    assert run.returncode == 0, run.stdout[-2000:] + run.stderr[-4000:]
    return run.stdout


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not installed")
def test_cache_under_sanitizers(tmp_path):
    exe = str(tmp_path / "cache_stress")
    cmd = ["g++", "-std=c++17", *SAN, "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
           "-I" + os.path.join(ROOT, "include"), "-I" + os.path.join(ROOT, "paper_2609_32278_amd", "csrc"),
           os.path.join(ROOT, "paper_2609_32278_amd", "csrc", "kvx_cache.cpp"),
           os.path.join(ROOT, "tests", "sanitize", "cache_stress.cpp"), "-o", exe]
    out = _build_and_run(cmd, exe, ["1000"], tmp_path)
    assert "passed" in out
    print(out)


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not installed")
def test_radix_tree_under_sanitizers(tmp_path):
    exe = str(tmp_path / "radix_stress")
    cmd = ["g++", "-std=c++17", *SAN, "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
           "-I" + os.path.join(ROOT, "include"), "-I" + os.path.join(ROOT, "paper_2609_32278_amd", "csrc"),
           os.path.join(ROOT, "paper_2609_32278_amd", "csrc", "kvx_radix.cpp"),
           os.path.join(ROOT, "tests", "sanitize", "radix_stress.cpp"), "-o", exe]
    out = _build_and_run(cmd, exe, ["200"], tmp_path)
    assert "passed" in out
    print(out)


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not installed")
def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_stress")
    cmd = ["gcc", "-std=c11", *SAN, "-fopenmp", os.path.join(ROOT, "oracle", "oracle.c"),
           os.path.join(ROOT, "tests", "sanitize", "oracle_stress.c"), "-lm", "-o", exe]
    out = _build_and_run(cmd, exe, ["300"], tmp_path)
    assert "passed" in out
    print(out)


@pytest.mark.skipif(shutil.which("g++") is None or not os.path.exists("/opt/rocm/lib/libamdhip64.so"),
                    reason="g++ or the HIP runtime library not installed")
def test_planner_under_sanitizers(tmp_path):
    exe = str(tmp_path / "plan_stress")
    cmd = ["g++", "-std=c++17", *SAN, "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
           "-I" + os.path.join(ROOT, "include"), "-I" + os.path.join(ROOT, "paper_2609_32278_amd", "csrc"),
           os.path.join(ROOT, "paper_2609_32278_amd", "csrc", "kvx_host.cpp"),
           os.path.join(ROOT, "tests", "sanitize", "plan_stress.cpp"),
           "-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib", "-o", exe]
    out = _build_and_run(cmd, exe, ["300"], tmp_path)
    assert "passed" in out
    print(out)

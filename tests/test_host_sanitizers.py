"""The host planner and step validator under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU only): tests/host/plan_check.cpp fuzzes valid steps, checks every plan's invariants and
the status codes of invalid steps. The C++ sources are built with g++ (no device code)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_planner_under_asan_ubsan(tmp_path):
    exe = tmp_path / "plan_check"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROOT, "paper_2608_15171_amd", "csrc"),
           os.path.join(ROOT, "paper_2608_15171_amd", "csrc", "plan.cpp"),
           os.path.join(ROOT, "tests", "host", "plan_check.cpp"), "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0 and r.stdout.strip() == "ok", (r.stdout + r.stderr)[-4000:]


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_c_abi_from_a_c_program(tmp_path):
    """include/ppas.h is a C header: a C11 program built with -Wall -Wextra -pedantic -Werror
    links libppas.so and calls its host-only entry points."""
    lib_dir = os.path.join(ROOT, "paper_2608_15171_amd")
    if not os.path.exists(os.path.join(lib_dir, "libppas.so")):
        pytest.skip("libppas.so not built")
    exe = tmp_path / "abi_from_c"
    cmd = ["gcc", "-std=c11", "-Wall", "-Wextra", "-pedantic", "-Werror", "-I", os.path.join(ROOT, "include"),
           os.path.join(ROOT, "tests", "host", "abi_from_c.c"), "-L", lib_dir, "-l:libppas.so",
           f"-Wl,-rpath,{lib_dir}", "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ)
    env["LD_LIBRARY_PATH"] = "/opt/rocm/lib:" + env.get("LD_LIBRARY_PATH", "")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 0 and r.stdout.strip() == "ok", (r.stdout + r.stderr)[-4000:]

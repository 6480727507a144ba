"""The C ABI from a C program on the GPU (tests/host/abi_gpu.c): device memory from
the HIP C API, ppas_kv_append and ppas_attn_step called without Python, checked
against the page-scatter rule and a closed-form attention result (equal value rows
give their value back exactly)."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_step_from_c(tmp_path):
    lib_dir = os.path.join(ROOT, "paper_2608_15171_amd")
    assert os.path.exists(os.path.join(lib_dir, "libppas.so")), "libppas.so not built"
    exe = tmp_path / "abi_gpu"
    cmd = ["gcc", "-std=c11", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__", "-I", "/opt/rocm/include",
           "-I", os.path.join(ROOT, "include"), os.path.join(ROOT, "tests", "host", "abi_gpu.c"),
           "-L", lib_dir, "-l:libppas.so", f"-Wl,-rpath,{lib_dir}", "-L", "/opt/rocm/lib", "-lamdhip64",
           "-Wl,-rpath,/opt/rocm/lib", "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    print("running the C program on the GPU", flush=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=90)
    assert r.returncode == 0 and r.stdout.strip() == "ok", (r.stdout + r.stderr)[-4000:]

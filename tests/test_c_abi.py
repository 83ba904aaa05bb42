"""The C ABI from a plain C program (tests/c/kvio_abi_demo.c) linked against
libkvio.so: host-side checks everywhere, a paged load/offload on the GPU."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2508_18572_amd")


def build_demo(tmp_path):
    exe = str(tmp_path / "kvio_abi_demo")
    subprocess.run(["gcc", "-std=c99", "-O1", "-Wall", "-Werror", "-D__HIP_PLATFORM_AMD__",
                    "-I", os.path.join(ROOT, "include"), "-I", "/opt/rocm/include",
                    os.path.join(ROOT, "tests", "c", "kvio_abi_demo.c"), "-o", exe,
                    "-L", PKG, "-lkvio", "-L", "/opt/rocm/lib", "-lamdhip64",
                    f"-Wl,-rpath,{PKG}", "-Wl,-rpath,/opt/rocm/lib"], check=True)
    return exe


def test_c_program_host_checks(tmp_path):
    exe = build_demo(tmp_path)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "host-only checks passed" in r.stdout


@pytest.mark.gpu
def test_c_program_gpu(tmp_path):
    exe = build_demo(tmp_path)
    r = subprocess.run([exe, "gpu"], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "gpu checks passed" in r.stdout

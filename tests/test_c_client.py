"""The library from plain C: include/estp.h compiled as C99 by gcc, linked against libestp.so and
the HIP runtime, with no Python in the loop (tests/c_abi/estp_c_client.c)."""
import os
import shutil
import subprocess

import pytest

import paper_2608_15592_amd as estp

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def _build(tmp_path) -> str:
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    lib_dir = os.path.dirname(os.path.abspath(estp.LIB_PATH))
    exe = str(tmp_path / "estp_c_client")
    cmd = ["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__", f"-I{ROCM}/include",
           f"-I{ROOT}/include", os.path.join(HERE, "c_abi", "estp_c_client.c"), "-o", exe, f"-L{lib_dir}", "-lestp",
           f"-L{ROCM}/lib", "-lamdhip64", "-lm", f"-Wl,-rpath,{lib_dir}", f"-Wl,-rpath,{ROCM}/lib"]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    return exe


def test_c_client_host_checks(tmp_path):
    exe = _build(tmp_path)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "host checks passed" in r.stdout


@pytest.mark.gpu
def test_c_client_gpu_closed_forms(tmp_path):
    exe = _build(tmp_path)
    r = subprocess.run([exe, "--gpu"], capture_output=True, text=True, timeout=120)
    print(r.stdout)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "gpu checks passed" in r.stdout

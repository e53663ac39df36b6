"""The host side of libestp under AddressSanitizer.

The library is rebuilt with -fsanitize=address on its host code only (argument validation,
workspace sizing, launch set-up, error messages; the gfx950 device code is built as usual),
then the host-only ABI tests run against it in a child process with the sanitizer runtime
preloaded.  An out-of-bounds access or use-after-free in that code aborts the child."""
import os
import subprocess
import sys

import pytest

from paper_2608_15592_amd import build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _gpu_present():
    import torch
    return torch.cuda.is_available()


@pytest.mark.skipif(_gpu_present(), reason="the host-validation cases use fake pointers")
def test_host_library_under_address_sanitizer(tmp_path):
    lib = build.build(out=str(tmp_path / "libestp_asan.so"), sanitize=True)
    env = dict(os.environ, LD_PRELOAD=build.asan_runtime(), ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               ESTP_LIBRARY=lib)
    probe = ("import paper_2608_15592_amd as e; e.load(); "
             "print(''.join(l for l in open('/proc/self/maps') if 'libestp' in l))")
    r = subprocess.run([sys.executable, "-c", probe], cwd=ROOT, env=env, capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr[-3000:]
    assert "libestp_asan.so" in r.stdout and "libestp.so" not in r.stdout.replace("libestp_asan.so", "")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-m", "not gpu", "-p", "no:cacheprovider",
                        "tests/test_abi.py", "tests/test_bench_cli.py"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert "AddressSanitizer" not in r.stderr

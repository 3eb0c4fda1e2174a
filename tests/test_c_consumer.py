"""The C ABI from plain C, without torch: tests/c_abi/abi_consumer.c is
compiled with gcc against include/wmtp.h and linked with libwmtp.so and the
HIP runtime.  On the CPU the build itself is the check (the header is valid
C11 and every call the program makes resolves in the library); on the GPU
the program runs the full, windowed and ring calls and checks closed forms
(K = 0 and V = 1: output exactly 1, lse = ln of the selected key count) and
the host-side argument errors."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "c_abi", "abi_consumer.c")
PKG = os.path.join(ROOT, "paper_2607_21535_amd")
LIB = os.path.join(PKG, "libwmtp.so")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def _build(out_dir):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not found")
    if not os.path.exists(LIB):
        pytest.skip("libwmtp.so is not built (python -m paper_2607_21535_amd.build)")
    exe = os.path.join(out_dir, "abi_consumer")
    cmd = ["gcc", "-std=c11", "-O1", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROCM, "include"), SRC, "-o", exe,
           "-L", PKG, "-lwmtp", "-L", os.path.join(ROCM, "lib"), "-lamdhip64", "-lm",
           f"-Wl,-rpath,{PKG}", f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}"]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr
    return exe


def test_c_program_builds_against_the_header(tmp_path):
    _build(str(tmp_path))


@pytest.mark.gpu
def test_c_program_runs_the_hot_path(tmp_path):
    exe = _build(str(tmp_path))
    print("running the C consumer of the ABI", flush=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    print(r.stdout, flush=True)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "0 failure(s)" in r.stdout

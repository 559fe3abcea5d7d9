"""The C ABI from plain C: tests/c_abi_check.c is compiled with the host C compiler
against include/prcr.h and the in-tree libprcr.so, and run as a child process.  It
checks, with no Python in between, that prefill capture, an IDENTITY revisit and
decode attention behave as their definitions fix (rebinding at the original
coordinates reproduces the prefill keys bit for bit; one-key attention returns the
value row)."""
import os
import shutil
import subprocess

import pytest

pytestmark = pytest.mark.gpu
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def test_plain_c_consumer(tmp_path):
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no host C compiler")
    lib = os.path.join(ROOT, "paper_2606_26631_amd")
    if not os.path.exists(os.path.join(lib, "libprcr.so")):
        pytest.fail("libprcr.so is not built")
    exe = str(tmp_path / "c_abi_check")
    cmd = [cc, "-std=c11", "-O1", "-Wall", "-D__HIP_PLATFORM_AMD__", f"-I{ROOT}/include",
           f"-I{ROCM}/include", os.path.join(ROOT, "tests", "c_abi_check.c"), f"-L{lib}", "-lprcr",
           f"-L{ROCM}/lib", "-lamdhip64", f"-Wl,-rpath,{lib}", f"-Wl,-rpath,{ROCM}/lib", "-o", exe]
    built = subprocess.run(cmd, capture_output=True, text=True, timeout=120)
    assert built.returncode == 0, built.stderr
    print("running the C consumer", flush=True)
    run = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    print(run.stdout, run.stderr, flush=True)
    assert run.returncode == 0, run.stderr
    assert "c_abi_check: ok" in run.stdout

"""The C ABI from a plain C program (gcc, no Python types): tests/abi_consumer.c.

Host-only calls: plan sizes for every (lmax, parity), the selection rules of
the reported paths, the orthonormality of the reported coupling coefficients,
the workspace size, the layer's buffer sizes and shape checks, and early
error returns.
"""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIBDIR = os.path.join(ROOT, "paper_2504_16068_amd")


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_c_consumer(tmp_path):
    if not os.path.exists(os.path.join(LIBDIR, "liballegro_tp.so")):
        pytest.skip("liballegro_tp.so not built (run __graft_entry__.build())")
    exe = tmp_path / "abi_consumer"
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-I", os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "tests", "abi_consumer.c"), "-L", LIBDIR, "-lallegro_tp",
                    "-Wl,-rpath," + LIBDIR, "-o", str(exe)], check=True)
    env = dict(os.environ)
    env["LD_LIBRARY_PATH"] = "/opt/rocm/lib:" + env.get("LD_LIBRARY_PATH", "")
    res = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=120)
    assert res.returncode == 0, res.stdout + res.stderr
    assert res.stdout.count("ok lmax=") == 6 and "ok layer" in res.stdout and "ok errors" in res.stdout

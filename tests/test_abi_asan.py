"""The host side of the library under AddressSanitizer (leak checking on).

The library's two HIP sources are compiled again with the sanitizer on their
host code only (each -fsanitize= behind -Xarch_host; the device code is built
as usual and never runs here), and the plain C consumer of the ABI
(tests/abi_consumer.c) runs against that build: plan creation and
destruction for every (lmax, parity), the coupling-table queries, workspace
and layer buffer sizes, and the early error returns.  Any heap overflow,
use after free or leak in those paths fails the test.
"""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2504_16068_amd", "csrc")
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
CLANG = "/opt/rocm/llvm/bin/clang"


@pytest.mark.skipif(not (os.path.exists(HIPCC) and os.path.exists(CLANG)), reason="ROCm toolchain not available")
def test_c_consumer_under_address_sanitizer(tmp_path):
    if not os.path.exists(os.path.join(CSRC, "generated", "tp_cores.inc")):
        pytest.skip("generated kernel sources missing (run __graft_entry__.build())")
    hip = [HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer",
           "-I", os.path.join(ROOT, "include"), "-I", CSRC]
    objs = []
    jobs = []
    for src in ("allegro_tp.hip", "allegro_layer.hip"):
        obj = str(tmp_path / src.replace(".hip", ".o"))
        objs.append(obj)
        jobs.append(subprocess.Popen(hip + ["-c", os.path.join(CSRC, src), "-o", obj],
                                     stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True))
    cg = str(tmp_path / "cg_builder.o")
    subprocess.run([CLANG + "++", "-O1", "-g", "-std=c++17", "-fPIC", "-fsanitize=address", "-I", CSRC, "-c",
                    os.path.join(CSRC, "cg_builder.cpp"), "-o", cg], check=True)
    for job in jobs:
        out, _ = job.communicate(timeout=600)
        assert job.returncode == 0, out[-2000:]
    lib = str(tmp_path / "liballegro_tp.so")
    subprocess.run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-Xarch_host", "-fsanitize=address",
                    *objs, cg, "-o", lib], check=True, capture_output=True)
    exe = str(tmp_path / "abi_consumer")
    subprocess.run([CLANG, "-std=c99", "-g", "-fsanitize=address", "-I", os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "tests", "abi_consumer.c"), "-L", str(tmp_path), "-lallegro_tp",
                    "-Wl,-rpath," + str(tmp_path), "-o", exe], check=True)
    env = dict(os.environ)
    env["LD_LIBRARY_PATH"] = "/opt/rocm/lib:" + env.get("LD_LIBRARY_PATH", "")
    env["ASAN_OPTIONS"] = "detect_leaks=1:halt_on_error=1:verify_asan_link_order=0"
    res = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert res.returncode == 0, (res.stdout + res.stderr)[-4000:]
    assert "ERROR: AddressSanitizer" not in res.stderr and "LeakSanitizer" not in res.stderr
    assert res.stdout.count("ok lmax=") == 6 and "ok layer" in res.stdout and "ok errors" in res.stdout

"""The C-ABI layer's host validation built with the address and undefined-behaviour
sanitizers (CPU): fs_api.cpp with host stubs of the kernel launchers (tests/asan), driven by
a C program that calls every entry point with valid and invalid arguments and checks each
status code. Any out-of-bounds access, leak or undefined behaviour aborts the run."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
       "-g", "-O1"]


@pytest.mark.skipif(shutil.which("g++") is None or shutil.which("gcc") is None,
                    reason="needs the GNU host compilers")
def test_abi_validation_under_sanitizers(tmp_path):
    inc = ["-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", "-I" + os.path.join(ROOT, "include")]
    src = os.path.join(ROOT, "paper_2609_32525_amd", "csrc", "fs_api.cpp")
    objs = []
    for cpp in (src, os.path.join(HERE, "asan", "abi_stubs.cpp")):
        o = str(tmp_path / (os.path.basename(cpp) + ".o"))
        subprocess.run(["g++", "-std=c++17", *inc, *SAN, "-c", cpp, "-o", o], check=True)
        objs.append(o)
    drv = str(tmp_path / "abi_driver.o")
    subprocess.run(["gcc", "-std=c11", *inc, *SAN, "-c", os.path.join(HERE, "asan", "abi_driver.c"),
                    "-o", drv], check=True)
    exe = str(tmp_path / "abi_driver")
    subprocess.run(["g++", *SAN, drv, *objs, "-o", exe], check=True)
    env = dict(os.environ,
               ASAN_OPTIONS="detect_leaks=1:abort_on_error=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    res = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    assert res.returncode == 0, res.stdout + res.stderr
    assert "all expectations hold" in res.stdout

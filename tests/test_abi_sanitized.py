"""The C ABI's host layer under AddressSanitizer and UndefinedBehaviorSanitizer.

tests/abi_host/abi_check.c is a C99 program that drives every entry point through its
argument checks (bad shapes and parameters, null, misaligned and short buffers, lists
given in part, empty layers), the status strings, the thread-local error message and,
with no GPU present, the CRISP_EHIP report of a call whose validation passes.  It is
linked here with api.cpp built by g++ under both sanitizers and with the kernel objects
of the normal build, and must exit cleanly with no sanitizer report.

Host only: it runs where no GPU is present, so that a call reaching a launch cannot
touch a device (its device pointers are fake addresses).
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_01925_amd", "csrc")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
SANITIZE = ["-fsanitize=address,undefined", "-fno-omit-frame-pointer", "-g", "-O1"]


def _skip_reason():
    if os.path.exists("/dev/kfd"):
        return "a GPU is present; this host-only check runs where no call can reach a device"
    if os.environ.get("LD_PRELOAD"):
        return "a preloaded library would come before the AddressSanitizer runtime"
    for tool in ("gcc", "g++"):
        if shutil.which(tool) is None:
            return f"{tool} not found"
    if not os.path.exists(os.path.join(ROCM, "lib", "libamdhip64.so")):
        return "HIP runtime library not found"
    return None


@pytest.mark.skipif(_skip_reason() is not None, reason=str(_skip_reason()))
def test_abi_host_layer_under_sanitizers(tmp_path):
    from paper_2609_01925_amd import build as B
    kernels = [os.path.join(B.BUILD, f) for f in ("estimate.o", "select.o", "attn.o")]
    if not all(os.path.exists(f) for f in kernels):
        B.build()
    api = tmp_path / "api_san.o"
    main = tmp_path / "abi_check.o"
    exe = tmp_path / "abi_check"
    steps = [
        ["g++", "-std=c++17", "-fPIC", *SANITIZE, "-D__HIP_PLATFORM_AMD__", f"-I{ROCM}/include",
         f"-I{B.INCLUDE}", f"-I{CSRC}", "-c", os.path.join(CSRC, "api.cpp"), "-o", str(api)],
        ["gcc", "-std=c99", "-Wall", "-Wextra", "-pedantic", "-Werror", *SANITIZE, f"-I{B.INCLUDE}", "-c",
         os.path.join(ROOT, "tests", "abi_host", "abi_check.c"), "-o", str(main)],
        ["g++", "-fsanitize=address,undefined", str(main), str(api), *kernels, f"-L{ROCM}/lib", "-lamdhip64",
         f"-Wl,-rpath,{ROCM}/lib", "-lpthread", "-o", str(exe)],
    ]
    for cmd in steps:
        p = subprocess.run(cmd, capture_output=True, text=True)
        assert p.returncode == 0, f"$ {' '.join(cmd)}\n{p.stdout}\n{p.stderr}"
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    p = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=120)
    assert p.returncode == 0, p.stdout + p.stderr
    assert "0 failures" in p.stdout and "runtime error" not in p.stderr and "AddressSanitizer" not in p.stderr, \
        p.stdout + p.stderr

"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer.

abi.hip (argument validation, workspace sizing, launch set-up) and
stack.hip (the stack executor) are rebuilt with both sanitizers on their host
side only, linked with the other objects of
the library build and with tests/sanitize/abi_fuzz.c, which calls every entry
point with edge-value arguments (see that file).  Runs only where no GPU is
present: there no call gets past its first HIP call, so the stand-in device
addresses are never used.
"""
import glob
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BUILD = os.path.join(ROOT, "paper_2608_09388_amd", "_build")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = os.path.join(ROCM, "bin", "hipcc")
CLANG = os.path.join(ROCM, "llvm", "bin", "clang")
CLANGXX = os.path.join(ROCM, "llvm", "bin", "clang++")


def test_abi_host_code_under_asan_ubsan(tmp_path):
    host = ("abi", "stack")    # sources whose host code is rebuilt with the sanitizers
    objs = [o for o in sorted(glob.glob(os.path.join(BUILD, "*.o")))
            if os.path.splitext(os.path.basename(o))[0] not in host]
    if not objs:
        pytest.skip("library objects not built (python -m paper_2608_09388_amd.build)")
    for tool in (HIPCC, CLANG, CLANGXX):
        if not os.path.exists(tool):
            pytest.skip(f"{tool} not found")
    inc = os.path.join(ROOT, "include")
    san = []
    for name in host:
        o = str(tmp_path / f"{name}_san.o")
        # host-side sanitizers only: each -fsanitize flag goes to the host compile
        subprocess.run([HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-fPIC", "-std=c++17", "-I",
                        inc, "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                        "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                        "-Xarch_host", "-fno-sanitize-recover=undefined",
                        "-Xarch_host", "-fno-omit-frame-pointer",
                        "-c", os.path.join(ROOT, "paper_2608_09388_amd", "csrc", f"{name}.hip"),
                        "-o", o], check=True, capture_output=True)
        san.append(o)
    fuzz_o = str(tmp_path / "fuzz.o")
    subprocess.run([CLANG, "-O1", "-g", "-fsanitize=address,undefined",
                    "-fno-sanitize-recover=undefined", "-D__HIP_PLATFORM_AMD__", "-I", inc,
                    "-I", os.path.join(ROCM, "include"),
                    "-c", os.path.join(ROOT, "tests", "sanitize", "abi_fuzz.c"), "-o", fuzz_o],
                   check=True, capture_output=True)
    exe = str(tmp_path / "abi_fuzz")
    subprocess.run([CLANGXX, "-fsanitize=address,undefined", fuzz_o, *san, *objs,
                    "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
                    "-Wl,-rpath," + os.path.join(ROCM, "lib"), "-o", exe],
                   check=True, capture_output=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([exe], env=env, capture_output=True, text=True, timeout=600)
    if r.returncode == 2 and "GPU is present" in r.stderr:
        pytest.skip("a GPU is present")
    assert r.returncode == 0, r.stdout + r.stderr
    assert "bad 0" in r.stdout
    calls = int(r.stdout.split()[1])
    assert calls >= 100000

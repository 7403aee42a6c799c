"""AddressSanitizer and UndefinedBehaviorSanitizer builds of the host code, on the CPU.

The oracle (gcc) and the library's host runtime (hipcc; the sanitizers act on
the host side only, the device code is built as usual) are compiled with
ASan + UBSan into a temporary directory, and the CPU suites that exercise them
run in a subprocess against those builds: the oracle's pins
(tests/test_oracle_pins.py) and the C ABI's host checks (tests/test_abi.py:
argument validation, scratch sizes, strerror, the device-less create).  Any
sanitizer report fails the test.  Nothing here runs on a GPU.
"""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=undefined",
       "-fno-omit-frame-pointer"]


def _run_suite(test_file, env_extra):
    env = dict(os.environ)
    env.update(env_extra)
    # the sanitizer runtime first; keep anything the environment preloads after it
    pre = env_extra["LD_PRELOAD"]
    if os.environ.get("LD_PRELOAD"):
        pre += ":" + os.environ["LD_PRELOAD"]
    env["LD_PRELOAD"] = pre
    env["ASAN_OPTIONS"] = "detect_leaks=0:verify_asan_link_order=0:abort_on_error=0"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-s", "-p", "no:cacheprovider", "-m",
                        "not gpu", test_file], env=env, capture_output=True, text=True,
                       cwd=ROOT, timeout=900)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "ERROR: AddressSanitizer" not in out, out[-4000:]
    assert "runtime error:" not in out, out[-4000:]
    assert " passed" in r.stdout
    return r.stdout


def test_oracle_pins_under_asan_and_ubsan(tmp_path):
    lib = str(tmp_path / "liboracle_san.so")
    subprocess.run(["gcc", "-O1", "-g"] + SAN + ["-fopenmp", "-fPIC", "-shared", "-fno-fast-math",
                    "-ffp-contract=off", "-o", lib, os.path.join(ROOT, "oracle", "kred_oracle.c"),
                    "-lm"], check=True)
    asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True,
                          text=True, check=True).stdout.strip()
    _run_suite("tests/test_oracle_pins.py", {"KRED_ORACLE_LIBRARY": lib, "LD_PRELOAD": asan})


def test_host_runtime_validation_under_asan_and_ubsan(tmp_path):
    from paper_2004_11127_amd import build as kbuild
    kernels = [os.path.join(kbuild.BUILD, os.path.splitext(s)[0] + ".o")
               for s in kbuild.SOURCES if s != "kred_api.cpp"]
    if not all(os.path.exists(o) for o in kernels):
        kbuild.build()
    obj = str(tmp_path / "kred_api_san.o")
    lib = str(tmp_path / "libkred_san.so")
    host_san = [f for s in SAN for f in ("-Xarch_host", s)]
    flags = [f for f in kbuild.FLAGS if f != "-O3"] + ["-O1", "-g"]
    subprocess.run([kbuild.HIPCC, "-x", "hip"] + flags + host_san +
                   ["-c", os.path.join(kbuild.CSRC, "kred_api.cpp"), "-o", obj], check=True)
    subprocess.run([kbuild.HIPCC, "-shared", "-fPIC", "--offload-arch=" + kbuild.ARCH,
                    "-shared-libsan"] + host_san + ["-o", lib, obj] + kernels, check=True)
    rt = glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")
    if not rt:
        pytest.skip("clang's ASan runtime is not installed")
    _run_suite("tests/test_abi.py", {"KRED_LIBRARY": lib, "LD_PRELOAD": rt[0]})

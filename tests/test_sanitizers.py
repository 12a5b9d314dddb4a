"""Host code under the address and undefined-behaviour sanitizers (CPU only; GPU code is never built with them):
the oracle's C (oracle/oracle.c) driven through every entry point, and the library's host layer
(csrc/dreams_api.hip: argument checks, planning, workspace sizes, status text) driven through calls that answer
or fail their checks without touching a device.  The drivers are in tests/sanitize/."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]


def _run(exe, tmp_path):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1",
               OMP_NUM_THREADS="4")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env, cwd=str(tmp_path))
    assert r.returncode == 0, r.stdout + r.stderr
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr
    return r.stdout


def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_driver")
    subprocess.run(["gcc", "-std=c11", "-O1", "-g", "-fopenmp"] + SAN +
                   [os.path.join(ROOT, "oracle", "oracle.c"), os.path.join(HERE, "oracle_driver.c"), "-o", exe, "-lm"],
                   check=True, capture_output=True, cwd=str(tmp_path))
    assert "oracle driver: ok" in _run(exe, tmp_path)


def test_host_layer_under_sanitizers(tmp_path):
    from paper_2606_00535_amd import build as B
    if not os.path.isdir(B.BUILD_DIR) or not all(
            os.path.exists(os.path.join(B.BUILD_DIR, os.path.basename(s) + ".o")) for s in B.sources()):
        B.build()
    hipcc = B.HIPCC
    if not os.path.exists(hipcc):
        pytest.skip("hipcc is not installed")
    san_host = []
    for flag in SAN:
        san_host += ["-Xarch_host", flag]     # host code only: the device code is built as usual
    api = os.path.join(B.CSRC, "dreams_api.hip")
    api_o = str(tmp_path / "api_san.o")
    cflags = [f for f in B.CFLAGS if f != "-O3"] + ["-O1", "-g"]
    subprocess.run([hipcc] + cflags + san_host + ["-c", api, "-o", api_o], check=True, capture_output=True)
    drv_o = str(tmp_path / "host_driver.o")
    subprocess.run([hipcc, "-O1", "-g", "-std=c++17"] + san_host +
                   ["-I" + B.INCLUDE, "-I/opt/rocm/include", "-D__HIP_PLATFORM_AMD__", "-c",
                    os.path.join(HERE, "host_driver.cpp"), "-o", drv_o], check=True, capture_output=True)
    objs = [os.path.join(B.BUILD_DIR, os.path.basename(s) + ".o") for s in B.sources()
            if os.path.basename(s) != "dreams_api.hip"]
    exe = str(tmp_path / "host_driver")
    subprocess.run([hipcc, "--offload-arch=" + B.ARCH] + san_host + ["-o", exe, drv_o, api_o] + objs,
                   check=True, capture_output=True)
    assert "host driver: ok" in _run(exe, tmp_path)

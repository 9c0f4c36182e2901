"""CPU builds with AddressSanitizer and UndefinedBehaviorSanitizer: the oracle
(every function on small and edge-sized inputs) and the C-ABI layer's host
validation and dispatch (cci_api.cpp linked against launcher stand-ins, so
no GPU is involved).  Any out-of-bounds access or undefined operation aborts
the driver with a report."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]


def _run(cmd, cwd):
    r = subprocess.run(cmd, cwd=cwd, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout}\n{r.stderr}"
    return r


@pytest.fixture(scope="module")
def build_dir(tmp_path_factory):
    return str(tmp_path_factory.mktemp("sanitize"))


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_oracle_under_sanitizers(build_dir):
    exe = os.path.join(build_dir, "oracle_driver")
    _run(["gcc", *SAN, "-std=c11", "-fopenmp", os.path.join(ROOT, "oracle", "cci_oracle.c"),
          os.path.join(HERE, "sanitize", "oracle_driver.c"), "-lm", "-o", exe], build_dir)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1", UBSAN_OPTIONS="print_stacktrace=1", OMP_NUM_THREADS="2")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=600, env=env)
    assert r.returncode == 0 and "oracle driver ok" in r.stdout, r.stdout + r.stderr


@pytest.mark.skipif(shutil.which("g++") is None or not os.path.isdir("/opt/rocm/include"), reason="needs g++ and HIP headers")
def test_abi_host_layer_under_sanitizers(build_dir):
    exe = os.path.join(build_dir, "abi_driver")
    src = [os.path.join(ROOT, "paper_1910_11971_amd", "csrc", "cci_api.cpp"),
           os.path.join(HERE, "sanitize", "host_stubs.cpp"), os.path.join(HERE, "sanitize", "abi_driver.cpp")]
    _run(["g++", *SAN, "-std=c++17", "-D__HIP_PLATFORM_AMD__", "-I", "/opt/rocm/include", "-I",
          os.path.join(ROOT, "include"), *src, "-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib", "-o", exe],
         build_dir)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=600, env=env)
    assert r.returncode == 0 and "abi driver ok" in r.stdout, r.stdout + r.stderr

"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

* The C ABI's argument validation (csrc/api.cpp, with the kernel launchers
  replaced by stubs that abort): tests/sanitize/abi_driver.cpp makes calls the
  library must reject on the host, including sizes whose naive products
  overflow; any launch reached, out-of-bounds access, signed overflow or leak
  fails the run.
* The oracle (oracle/hatq_oracle.c): tests/sanitize/oracle_driver.c runs every
  stage on small random layers of each kind (DH/WH, small-cin, transposed, 1x1,
  padded Paley orders).
Both are built with g++/gcc and -fsanitize=address,undefined (host code only).
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-O1", "-g"]
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def _run(exe, tmp_path):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", OMP_NUM_THREADS="4")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300, cwd=tmp_path)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "runtime error" not in r.stderr and "ERROR: AddressSanitizer" not in r.stderr, r.stderr


@pytest.mark.skipif(shutil.which("g++") is None or not os.path.exists(f"{ROCM}/include/hip/hip_runtime.h"),
                    reason="needs g++ and the HIP headers")
def test_abi_validation_sanitized(tmp_path):
    exe = str(tmp_path / "abi_san")
    cmd = ["g++", "-std=c++17", "-D__HIP_PLATFORM_AMD__", f"-I{ROCM}/include", f"-I{ROOT}/include", *SAN,
           f"{ROOT}/paper_2608_01653_amd/csrc/api.cpp", f"{ROOT}/tests/sanitize/abi_stubs.cpp",
           f"{ROOT}/tests/sanitize/abi_driver.cpp", f"-L{ROCM}/lib", "-lamdhip64", f"-Wl,-rpath,{ROCM}/lib",
           "-o", exe]
    subprocess.run(cmd, check=True, capture_output=True, timeout=300)
    _run(exe, tmp_path)


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_oracle_sanitized(tmp_path):
    exe = str(tmp_path / "orc_san")
    cmd = ["gcc", "-std=c11", "-fopenmp", "-ffp-contract=off", *SAN, f"{ROOT}/oracle/hatq_oracle.c",
           f"{ROOT}/tests/sanitize/oracle_driver.c", "-lm", "-o", exe]
    subprocess.run(cmd, check=True, capture_output=True, timeout=300)
    _run(exe, tmp_path)

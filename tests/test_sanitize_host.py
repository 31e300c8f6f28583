"""The host layer and the oracle under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

Builds tests/sanitize/driver.cpp with the C-ABI host sources (budget allocation, offsets, argument
validation) and the oracle's C source, all compiled by gcc/g++ with -fsanitize=address,undefined and
linked against the HIP host runtime, then runs it: allocation results must equal the oracle's on
seeded random problems, every validation path must return its status, and the sanitizers must
report nothing (any report aborts the run).
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_03235_amd", "csrc")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]


def _gpu():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


@pytest.mark.skipif(shutil.which("g++") is None or not os.path.exists("/opt/rocm/lib/libamdhip64.so"),
                    reason="needs g++ and the HIP host runtime")
@pytest.mark.skipif(_gpu(), reason="host-only run: the device entry points are driven through validation only")
def test_host_and_oracle_under_sanitizers(tmp_path):
    cxx = ["g++", "-std=c++17", *SAN, "-ffp-contract=off", "-fno-fast-math", "-D__HIP_PLATFORM_AMD__",
           "-isystem", "/opt/rocm/include", "-I", os.path.join(ROOT, "include"), "-I", CSRC]
    objs = []
    for src in (os.path.join(CSRC, "sgdkv_host.cpp"), os.path.join(CSRC, "profile.cpp"),
                os.path.join(ROOT, "tests", "sanitize", "launch_stubs.cpp"),
                os.path.join(ROOT, "tests", "sanitize", "driver.cpp")):
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        subprocess.run([*cxx, "-c", src, "-o", obj], check=True)
        objs.append(obj)
    orc = str(tmp_path / "oracle.o")
    subprocess.run(["gcc", "-std=c11", *SAN, "-ffp-contract=off", "-fno-fast-math", "-c",
                    os.path.join(ROOT, "oracle", "sgdkv_oracle.c"), "-o", orc], check=True)
    exe = str(tmp_path / "driver")
    subprocess.run(["g++", *SAN, *objs, orc, "-o", exe, "-L/opt/rocm/lib", "-Wl,-rpath,/opt/rocm/lib",
                    "-lamdhip64", "-lm"], check=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0, f"sanitizer run failed (rc {r.returncode}):\n{r.stdout[-3000:]}\n{r.stderr[-6000:]}"
    assert "SANITIZE PASS" in r.stdout

"""The host layer (argument validation, workspace sizing, launch planning) built
for the CPU with g++ under AddressSanitizer and UndefinedBehaviorSanitizer
against stub launchers (tests/host/stubs.cpp), and driven by a seeded
descriptor fuzzer (tests/host/fuzz_desc.cpp): random and near-valid
descriptors, null / misaligned / aligned pointers and workspace sizes around
the reported one. Any sanitizer finding aborts the run; a call that fails must
not have launched anything, and every launch's arguments must be consistent."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ROCM_INCLUDE = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "include")
SOURCES = ["tests/host/fuzz_desc.cpp", "tests/host/stubs.cpp",
           "paper_2006_03555_amd/csrc/favor_api.cpp", "paper_2006_03555_amd/csrc/timing.cpp"]


@pytest.fixture(scope="module")
def fuzzer(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None or not os.path.isdir(os.path.join(ROCM_INCLUDE, "hip")):
        pytest.skip("needs g++ and the HIP headers")
    exe = str(tmp_path_factory.mktemp("host") / "fuzz_desc")
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer",
           "-D__HIP_PLATFORM_AMD__", "-I", ROCM_INCLUDE, "-I", os.path.join(ROOT, "include"),
           *[os.path.join(ROOT, s) for s in SOURCES], "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    return exe


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_descriptor_fuzz_under_sanitizers(fuzzer, seed):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([fuzzer, str(seed), "20000"], capture_output=True, text=True, env=env,
                       timeout=300)
    assert r.returncode == 0, (r.stdout + r.stderr)[-3000:]
    assert "0 failures" in r.stdout

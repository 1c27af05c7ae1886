"""The library's host code under sanitizers, on the CPU.

* tests/native/host_checks.cpp, built with g++ -fsanitize=address,undefined
  from the host sources of libnsp (validation, unit schedule, recompute plan,
  SP-tree planner, executor and entry-point argument checks) with the kernel
  launchers stubbed out, runs seeded random and malformed work lists through
  the C ABI on a machine without a GPU.
* tests/native/cache_stress.cpp drives the schedule cache from four threads
  through many more keys than it holds, under ThreadSanitizer and under
  AddressSanitizer (an entry freed while still held, or an unlocked access,
  is reported).
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_22755_amd", "csrc")
NATIVE = os.path.join(ROOT, "tests", "native")
ROCM = "/opt/rocm"

pytestmark = pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")


def _build(out, sources, flags, libs=()):
    cmd = ["g++", "-std=c++17", "-O1", "-g", *flags, "-fno-sanitize-recover=all", "-ffp-contract=off",
           "-I", os.path.join(ROOT, "include"), "-I", CSRC, *sources, "-o", out, *libs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]


def _run(exe, env_extra):
    env = dict(os.environ, **env_extra)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=600, env=env)
    return r.returncode, r.stdout, r.stderr


@pytest.mark.timeout(900)
def test_host_code_under_asan_ubsan(tmp_path):
    if not os.path.exists(os.path.join(ROCM, "include", "hip", "hip_runtime.h")):
        pytest.skip("HIP headers not available")
    import torch
    if torch.cuda.device_count() > 0:
        pytest.skip("the host checks run on a machine without a GPU")
    exe = str(tmp_path / "host_checks")
    srcs = [os.path.join(NATIVE, "host_checks.cpp"), os.path.join(NATIVE, "launch_stubs.cpp")]
    srcs += [os.path.join(CSRC, f) for f in ("nsp_abi.cpp", "planner.cpp", "executor.cpp")]
    _build(exe, srcs, ["-fsanitize=address,undefined", "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROCM, "include"),
                       "-Wno-unknown-pragmas"],
           libs=["-L", os.path.join(ROCM, "lib"), "-lamdhip64", f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}"])
    rc, out, err = _run(exe, {"ASAN_OPTIONS": "detect_leaks=0", "UBSAN_OPTIONS": "print_stacktrace=1"})
    assert rc == 0 and "host checks ok" in out, (out + err)[-4000:]
    assert "runtime error" not in err and "AddressSanitizer" not in err, err[-4000:]


@pytest.mark.timeout(600)
@pytest.mark.parametrize("san", ["thread", "address,undefined"])
def test_schedule_cache_concurrent_eviction(tmp_path, san):
    exe = str(tmp_path / "cache_stress")
    _build(exe, [os.path.join(NATIVE, "cache_stress.cpp")], [f"-fsanitize={san}", "-pthread"])
    rc, out, err = _run(exe, {"TSAN_OPTIONS": "halt_on_error=1", "ASAN_OPTIONS": "detect_leaks=1"})
    assert rc == 0 and "cache stress ok" in out, (out + err)[-4000:]
    assert "WARNING: ThreadSanitizer" not in err and "AddressSanitizer" not in err, err[-4000:]

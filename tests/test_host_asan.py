"""The library's host C++ under AddressSanitizer and UBSan (CPU only).

Builds api.hip and control.hip with the sanitizers on their host code
(device code is compiled as usual), links them with stand-ins for the kernel
launchers and a driver (tests/asan/host_driver.cpp) that runs the metadata
lowering, the transition-list checks, the controller and the argument and
pointer checks of the device entry points on exact-size heap arrays, and
requires a clean run: no sanitizer report, every call's status as
documented."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_33536_amd", "csrc")
INCLUDE = os.path.join(ROOT, "include")
HERE = os.path.join(ROOT, "tests", "asan")


def _run(cmd, cwd):
    p = subprocess.run(cmd, cwd=cwd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in p.stdout.splitlines() if "packed-fp32-ops" not in l)
    assert p.returncode == 0, f"{' '.join(cmd[:3])}...: {out[-3000:]}"
    return out


def test_host_code_clean_under_address_sanitizer(tmp_path):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    gxx = shutil.which("g++")
    if not os.path.exists(hipcc) or not gxx:
        pytest.skip("hipcc or g++ missing")
    host_san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                "-Xarch_host", "-fno-omit-frame-pointer"]
    common = ["-O1", "-g", "-fPIC", "-std=c++17", f"-I{INCLUDE}", f"-I{CSRC}"]
    for src in ("api.hip", "control.hip"):
        _run([hipcc, "--offload-arch=gfx950", *common, *host_san, "-Xclang", "-target-feature", "-Xclang",
              "-packed-fp32-ops", "-c", os.path.join(CSRC, src), "-o", src.replace(".hip", ".o")], tmp_path)
    gflags = ["-O1", "-g", "-std=c++17", "-fsanitize=address,undefined", "-fno-omit-frame-pointer",
              "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", f"-I{INCLUDE}", f"-I{CSRC}"]
    for src in ("launch_stubs.cpp", "host_driver.cpp"):
        _run([gxx, *gflags, "-c", os.path.join(HERE, src), "-o", src.replace(".cpp", ".o")], tmp_path)
    _run([gxx, "-fsanitize=address,undefined", "host_driver.o", "api.o", "control.o", "launch_stubs.o",
          "-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib", "-o", "host_driver"], tmp_path)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", HIP_VISIBLE_DEVICES="")
    p = subprocess.run([str(tmp_path / "host_driver")], cwd=tmp_path, env=env, stdout=subprocess.PIPE,
                       stderr=subprocess.STDOUT, text=True, timeout=300)
    assert p.returncode == 0 and "host driver ok" in p.stdout, p.stdout[-4000:]
    assert "runtime error" not in p.stdout and "AddressSanitizer" not in p.stdout, p.stdout[-4000:]

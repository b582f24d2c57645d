"""The host side of the library under AddressSanitizer and UndefinedBehavior-
Sanitizer: the host sources (C ABI, planner, schedule generator) are built
with g++ -fsanitize=address,undefined and linked with the regular device
object into a second copy of the library; the C-ABI tests then run against
it in a child process with the sanitizer runtimes preloaded. Any report
(memory error, undefined behaviour) ends that process with an error.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2607_08754_amd")
CSRC = os.path.join(PKG, "csrc")
HOST_SOURCES = ["api.cpp", "plan.cpp", "pe_schedule.cpp"]


def _runtime(name):
    out = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return out if os.path.isabs(out) and os.path.exists(out) else None


def test_abi_tests_under_sanitizers(tmp_path):
    if shutil.which("g++") is None:
        pytest.skip("g++ not available")
    asan, ubsan = _runtime("libasan.so"), _runtime("libubsan.so")
    if not asan or not ubsan:
        pytest.skip("sanitizer runtimes not available")
    kobj = os.path.join(PKG, "_build", "kernels.o")
    if not os.path.exists(kobj):
        from paper_2607_08754_amd.build import build
        build()
    objs = []
    for src in HOST_SOURCES:
        obj = str(tmp_path / (os.path.splitext(src)[0] + ".o"))
        cmd = ["g++", "-std=c++17", "-O1", "-g", "-fPIC", "-fno-omit-frame-pointer",
               "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-D__HIP_PLATFORM_AMD__",
               "-I/opt/rocm/include", "-I", os.path.join(ROOT, "include"), "-I", CSRC,
               "-c", os.path.join(CSRC, src), "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-4000:]
        objs.append(obj)
    lib = str(tmp_path / "libslorr_sanitized.so")
    r = subprocess.run(["g++", "-shared", "-fsanitize=address,undefined", *objs, kobj, "-L/opt/rocm/lib",
                        "-lamdhip64", f"-Wl,--version-script={os.path.join(CSRC, 'exports.map')}", "-o", lib],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ)
    env.update({"LD_PRELOAD": f"{asan}:{ubsan}", "SLORR_LIB": lib,
                "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1",
                "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"})
    # -s: a report goes straight to the child's stderr (pytest's capture would
    # drop it when the sanitizer ends the process)
    r = subprocess.run([sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", "test_abi_cpu.py"),
                        "-x", "-q", "-s", "-p", "no:cacheprovider"], cwd=ROOT, env=env,
                       capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    print(out[-2000:])
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-6000:]
    assert r.returncode == 0 and " passed" in out, out[-6000:]

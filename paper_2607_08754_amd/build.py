"""Build libslorr.so (HIP for gfx950 + host C++) in-tree with hipcc.

    python -m paper_2607_08754_amd.build            # the library
    python -m paper_2607_08754_amd.build --probe    # + the main-loop ceiling probe

Objects go to paper_2607_08754_amd/_build/, the library to
paper_2607_08754_amd/libslorr.so (replaced atomically), the diagnostic
program csrc/probe_ceiling.hip to paper_2607_08754_amd/probe_ceiling.
"""
from __future__ import annotations

import os
import re
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libslorr.so")
PROBE = os.path.join(PKG, "probe_ceiling")

SOURCES = ["kernels.hip", "api.cpp", "plan.cpp", "pe_schedule.cpp"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

COMMON = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    # keep the compiler from forming packed fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE, "-I", CSRC, "-Wall", "-Wno-unused-result", "-fvisibility=hidden",
]


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *COMMON, "-c", os.path.join(CSRC, src), "-o", obj]
    if src.endswith(".hip"):
        cmd.append("-Rpass-analysis=kernel-resource-usage")
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{res.stdout}\n{res.stderr}")
    if src.endswith(".hip"):
        # a kernel whose private arrays or registers went to scratch memory
        # runs several times slower: refuse the build
        name, bad = None, []
        for line in res.stderr.splitlines():
            m = re.search(r"Function Name: (\S+)", line)
            if m:
                name = m.group(1)
            m = re.search(r"ScratchSize \[bytes/lane\]: (\d+)", line)
            if m and int(m.group(1)) > 0:
                bad.append(f"{name}: {m.group(1)} bytes/lane")
        if bad:
            raise RuntimeError("kernels use scratch memory:\n" + "\n".join(bad))
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(max_workers=min(4, len(SOURCES))) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs,
           f"-Wl,--version-script={os.path.join(CSRC, 'exports.map')}", "-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed:\n{res.stdout}\n{res.stderr}")
    # a kernel whose host stub went missing would only fail at dlopen time
    und = subprocess.run(["nm", "-u", "--demangle", tmp], capture_output=True, text=True).stdout
    bad = [l for l in und.splitlines() if "slorr" in l]
    if bad:
        raise RuntimeError("undefined library symbols:\n" + "\n".join(bad))
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


def build_probe(verbose: bool = False) -> str:
    cmd = [HIPCC, *COMMON, os.path.join(CSRC, "probe_ceiling.hip"), "-o", PROBE + ".tmp"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed on probe_ceiling.hip:\n{res.stdout}\n{res.stderr}")
    os.replace(PROBE + ".tmp", PROBE)
    if verbose:
        print(f"built {PROBE}")
    return PROBE


if __name__ == "__main__":
    build(verbose=True)
    if "--probe" in sys.argv[1:]:
        build_probe(verbose=True)
    sys.exit(0)

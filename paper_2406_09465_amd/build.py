"""Builds libkorch.so (host library + gfx950 helper kernels) in-tree.

Host C++ sources are compiled with g++ against the HIP runtime headers, the
HIP source with hipcc for gfx950, and everything is linked with hipcc.  The
runtime compiler helper `korch_rtc` (csrc/tools) is built next to the library.  The
device prelude that generated kernels include at run time is embedded into
the library as a string.

Usage:  python -m paper_2406_09465_amd.build   (or build() from Python)
"""

from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libkorch.so")
RTC_HELPER = os.path.join(PKG, "korch_rtc")  # runtime compiler, run by the library as a child process
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = os.path.join(ROCM, "bin", "hipcc")

HIP_FLAGS = ["--offload-arch=gfx950", "-O3", "-fPIC", "-std=c++17",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
CXX_FLAGS = ["-O2", "-fPIC", "-std=c++17", "-Wall", "-Wno-unused-function", "-Wno-unused-result",
             "-D__HIP_PLATFORM_AMD__", f"-I{ROCM}/include"]


def _embed_device_sources():
    src = open(os.path.join(CSRC, "device", "prelude.h")).read()
    if ")KORCHSRC\"" in src:
        raise RuntimeError("delimiter collision in device prelude")
    out = os.path.join(BUILD, "device_src.cpp")
    text = ("// generated from csrc/device/prelude.h\nnamespace korch {\n"
            f"extern const char* k_device_prelude;\nconst char* k_device_prelude = R\"KORCHSRC({src})KORCHSRC\";\n}}\n")
    if not os.path.exists(out) or open(out).read() != text:
        with open(out, "w") as f:
            f.write(text)
    return out


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("command failed: " + " ".join(cmd) + "\n" + r.stdout + r.stderr)
    return r


def build(verbose: bool = False, jobs: int = 8) -> str:
    """Compile every source and link libkorch.so; returns the library path."""
    os.makedirs(BUILD, exist_ok=True)
    inc = [f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}"]
    jobs_list = []
    for name in sorted(os.listdir(CSRC)):
        path = os.path.join(CSRC, name)
        if name.endswith(".cpp"):
            obj = os.path.join(BUILD, name[:-4] + ".o")
            jobs_list.append(["g++", *CXX_FLAGS, *inc, "-c", path, "-o", obj])
        elif name.endswith(".hip"):
            obj = os.path.join(BUILD, name[:-4] + ".hip.o")
            jobs_list.append([HIPCC, *HIP_FLAGS, *inc, "-c", path, "-o", obj])
    emb = _embed_device_sources()
    jobs_list.append(["g++", *CXX_FLAGS, "-c", emb, "-o", os.path.join(BUILD, "device_src.o")])
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        for r in ex.map(_run, jobs_list):
            if verbose and (r.stdout or r.stderr):
                print(r.stdout, r.stderr, file=sys.stderr)
    objs = [c[-1] for c in jobs_list]
    tmp = LIB + ".tmp"
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, f"-L{ROCM}/lib", "-ldl",
          f"-Wl,-rpath,{ROCM}/lib", "-o", tmp])
    os.replace(tmp, LIB)
    tmp = RTC_HELPER + ".tmp"
    _run(["g++", "-O2", "-std=c++17", "-Wall", "-D__HIP_PLATFORM_AMD__", f"-I{ROCM}/include",
          os.path.join(CSRC, "tools", "korch_rtc.cpp"), "-ldl", "-o", tmp])
    os.replace(tmp, RTC_HELPER)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))

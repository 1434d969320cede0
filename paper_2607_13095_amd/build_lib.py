"""Build libhswa.so (the HIP kernels and the C ABI) in-tree for gfx950.

    python -m paper_2607_13095_amd.build_lib

Each ``csrc/*.hip`` file is compiled with hipcc (and each host-only
``csrc/*.cpp`` file with the host C++ compiler) to an object under ``_build/``;
the objects are linked into ``libhswa.so`` next to this file.
"""

from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libhswa.so")
SOURCES = ["api.hip", "kv_append.hip", "decode.hip", "prefill.hip", "prefill_window.hip", "prefill_run.hip", "noalloc.hip", "decode_append.hip"]
HOST_SOURCES = ["allocator.cpp", "prefix_tree.cpp"]
CXX = os.environ.get("CXX", shutil.which("g++") or "g++")
CXXFLAGS = ["-O2", "-std=c++17", "-fPIC", "-Wall", "-I", os.path.join(ROOT, "include")]
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", shutil.which("hipcc") or "/opt/rocm/bin/hipcc")
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
    "-I", os.path.join(ROOT, "include"),
    # no packed fp32 instructions (v_pk_*_f32) anywhere in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass does not know the packed-fp32 target feature; that warning is harmless
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in r.stderr.splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{err}")
    return err


def build(verbose: bool = False) -> str:
    """Compile every source and link libhswa.so; returns the library path."""
    os.makedirs(BUILD, exist_ok=True)
    objs = [os.path.join(BUILD, s.replace(".hip", ".o")) for s in SOURCES]
    cmds = [[HIPCC, *FLAGS, "-c", os.path.join(CSRC, s), "-o", o] for s, o in zip(SOURCES, objs)]
    host_objs = [os.path.join(BUILD, s.replace(".cpp", ".host.o")) for s in HOST_SOURCES]
    cmds += [[CXX, *CXXFLAGS, "-c", os.path.join(CSRC, s), "-o", o] for s, o in zip(HOST_SOURCES, host_objs)]
    objs += host_objs
    with cf.ThreadPoolExecutor(max_workers=min(len(cmds), 8)) as ex:
        for err in ex.map(_run, cmds):
            if verbose and err.strip():
                print(err, file=sys.stderr)
    tmp = LIB + ".tmp"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs])
    os.replace(tmp, LIB)
    return LIB


# Host-sanitizer build: the host code (the C ABI's validation in api.hip, the
# allocator, the prefix tree) under gcc's address and undefined-behaviour
# sanitizers, linked with the device objects of build(). Load it with the
# sanitizer runtimes preloaded (sanitizer_env) and HSWA_LIB naming it.
SAN_FLAGS = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
             "-fno-sanitize-recover=undefined"]
HIP_HOST_FLAGS = ["-D__HIP_PLATFORM_AMD__", "-I", "/opt/rocm/include"]


def build_host_sanitized(out_dir: str) -> str:
    """Build libhswa_san.so in out_dir; returns its path."""
    dev_objs = [os.path.join(BUILD, s.replace(".hip", ".o")) for s in SOURCES if s != "api.hip"]
    if not all(os.path.exists(o) for o in dev_objs):
        build()
    os.makedirs(out_dir, exist_ok=True)
    # api.hip holds host code only; a one-line wrapper lets the host compiler take it as C++
    wrap = os.path.join(out_dir, "api_host.cpp")
    with open(wrap, "w") as f:
        f.write(f'#include "{os.path.join(CSRC, "api.hip")}"\n')
    units = [(wrap, HIP_HOST_FLAGS)] + [(os.path.join(CSRC, s), []) for s in HOST_SOURCES]
    objs = []
    for src, extra in units:
        o = os.path.join(out_dir, os.path.basename(src) + ".san.o")
        _run([CXX, "-std=c++17", "-fPIC", *SAN_FLAGS, *extra, "-I", os.path.join(ROOT, "include"), "-c", src, "-o", o])
        objs.append(o)
    lib = os.path.join(out_dir, "libhswa_san.so")
    _run([CXX, "-shared", *SAN_FLAGS, "-o", lib, *objs, *dev_objs, "-L/opt/rocm/lib", "-lamdhip64",
          "-Wl,-rpath,/opt/rocm/lib"])
    return lib


def sanitizer_env(lib: str) -> dict:
    """Environment that runs Python with the sanitizer runtimes preloaded and
    the binding loading `lib`."""
    rt = [subprocess.run([CXX, f"-print-file-name={n}"], capture_output=True, text=True).stdout.strip()
          for n in ("libasan.so", "libubsan.so")]
    env = dict(os.environ)
    env.update(LD_PRELOAD=" ".join(rt), HSWA_LIB=lib, ASAN_OPTIONS="detect_leaks=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    return env


if __name__ == "__main__":
    print(build(verbose=True))

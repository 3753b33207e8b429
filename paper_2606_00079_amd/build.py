"""Builds libbitsmoe.so in-tree: hipcc for the gfx950 kernels, g++ for the host
code, one shared library next to this file.

    python -m paper_2606_00079_amd.build              # build (always recompiles)
    python -m paper_2606_00079_amd.build --sanitize   # host-instrumented copy

``--sanitize`` builds libbitsmoe_san.so: the same sources with the host code
(every .cpp, and the host side of every .hip) instrumented by AddressSanitizer
and UndefinedBehaviorSanitizer, all with the ROCm clang so that one sanitizer
runtime serves both; device code is built as usual.  Load it in a process
that preloads that runtime, e.g.

    LD_PRELOAD=$(python -m paper_2606_00079_amd.build --asan-runtime) \
    ASAN_OPTIONS=detect_leaks=0 BITSMOE_LIB=paper_2606_00079_amd/libbitsmoe_san.so \
    python -m pytest tests/test_abi.py
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libbitsmoe.so")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
ARCH = "gfx950"

HIP_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++20", "-fPIC", "-ffp-contract=off",
    # packed fp32 VALU ops are kept out of the device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-command-line-argument",
]
CXX_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-ffp-contract=off", "-D__HIP_PLATFORM_AMD__",
             f"-I{ROCM}/include"]


def _hipcc() -> str:
    p = os.path.join(ROCM, "bin", "hipcc")
    return p if os.path.exists(p) else "hipcc"


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError("build failed: " + " ".join(cmd) + "\n" + out)
    return out


def sources():
    hip = sorted(f for f in os.listdir(CSRC) if f.endswith(".hip"))
    cpp = sorted(f for f in os.listdir(CSRC) if f.endswith(".cpp"))
    return hip, cpp


SAN_LIB = os.path.join(PKG, "libbitsmoe_san.so")
SAN_BUILD = os.path.join(ROOT, "_build_san")
# host-side sanitizers only: on hipcc lines each one follows -Xarch_host
SAN_HOST = ["-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=undefined"]


def asan_runtime() -> str:
    """The ROCm clang's shared AddressSanitizer runtime (to preload)."""
    import glob
    c = sorted(glob.glob(os.path.join(ROCM, "llvm", "lib", "clang", "*", "lib", "linux",
                                      "libclang_rt.asan-x86_64.so")))
    if not c:
        raise FileNotFoundError("no libclang_rt.asan-x86_64.so under " + ROCM)
    return c[-1]


def build(verbose: bool = False, jobs: int = 8, sanitize: bool = False) -> str:
    bdir, lib = (SAN_BUILD, SAN_LIB) if sanitize else (BUILD, LIB)
    os.makedirs(bdir, exist_ok=True)
    hip, cpp = sources()
    cmds = []
    objs = []
    hip_san = [x for f in SAN_HOST for x in ("-Xarch_host", f)] + ["-g"] if sanitize else []
    for f in hip:
        o = os.path.join(bdir, f + ".o")
        cmds.append([_hipcc(), *HIP_FLAGS, *hip_san, f"-I{INCLUDE}", f"-I{CSRC}", "-c",
                     os.path.join(CSRC, f), "-o", o])
        objs.append(o)
    if sanitize:
        cxx = os.path.join(ROCM, "llvm", "bin", "clang++")
        cxx_flags = [*CXX_FLAGS, *SAN_HOST, "-g", "-fno-omit-frame-pointer"]
    else:
        cxx = shutil.which("g++") or "c++"
        cxx_flags = CXX_FLAGS
    for f in cpp:
        o = os.path.join(bdir, f + ".o")
        cmds.append([cxx, *cxx_flags, f"-I{INCLUDE}", f"-I{CSRC}", "-c",
                     os.path.join(CSRC, f), "-o", o])
        objs.append(o)
    with ThreadPoolExecutor(max(1, min(jobs, len(cmds)))) as ex:
        outs = list(ex.map(_run, cmds))
    if verbose:
        for c, o in zip(cmds, outs):
            print(" ".join(c))
            if o.strip():
                print(o)
    tmp = lib + ".tmp"
    link_san = [x for f in SAN_HOST for x in ("-Xarch_host", f)] + ["-shared-libasan"] if sanitize else []
    _run([_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *link_san, "-o", tmp, *objs,
          f"-L{ROCM}/lib", "-lamdhip64", "-ldl"])
    # A kernel whose host stub was dropped links fine but fails at load time.
    nm = shutil.which("nm")
    if nm:
        undef = _run([nm, "-u", tmp])
        missing = [l for l in undef.splitlines() if "__device_stub__" in l]
        if missing:
            raise RuntimeError("kernel host stubs missing from the library:\n" + "\n".join(missing))
    os.replace(tmp, lib)
    return lib


if __name__ == "__main__":
    if "--asan-runtime" in sys.argv:
        print(asan_runtime())
    else:
        print(build(verbose="-v" in sys.argv, sanitize="--sanitize" in sys.argv))

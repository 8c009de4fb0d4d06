"""Builds libsf_decode_attn.so for gfx950 with hipcc, in-tree.

    python -m paper_2601_12784_amd.build
    python -m paper_2601_12784_amd.build --sanitize [--run-tests]

--sanitize builds a CPU-test copy, _build_san/libsf_decode_attn_san.so,
whose host sources (planner, page pool, cost model, extend planner, runner,
C entry points) are compiled by g++ with AddressSanitizer and
UndefinedBehaviorSanitizer (errors abort); the kernels are built as usual,
without instrumentation. --run-tests then runs the CPU test tier
(pytest -m "not gpu") against that copy, with the sanitizer runtimes
preloaded into the interpreter.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libsf_decode_attn.so")
SOURCES = ["plan.cpp", "pages.cpp", "cost.cpp", "extend.cpp", "runner.cpp", "api.cpp", "decode_attn.hip", "extend_attn.hip", "probe.hip",
           "scratch.hip"]
ARCH = "gfx950"

# -packed-fp32-ops: keep the compiler from forming packed fp32 VALU ops.
HIP_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-command-line-argument",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found; the HIP library cannot be built")


def build(verbose: bool = False) -> str:
    """Compiles every source and links the shared library (always rebuilds)."""
    cc = hipcc()
    objdir = os.path.join(PKG, "_build")
    os.makedirs(objdir, exist_ok=True)
    objs = []
    for src in SOURCES:
        obj = os.path.join(objdir, src + ".o")
        cmd = [cc, *HIP_FLAGS, "-I", INCLUDE, "-I", CSRC, "-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)
        objs.append(obj)
    tmp = LIB + ".tmp"
    cmd = [cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


HOST_SOURCES = [s for s in SOURCES if s.endswith(".cpp")]
SAN_DIR = os.path.join(PKG, "_build_san")
SAN_LIB = os.path.join(SAN_DIR, "libsf_decode_attn_san.so")
SAN_FLAGS = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]


def build_sanitized(verbose: bool = False) -> str:
    """The CPU-test copy described in the module docstring."""
    os.makedirs(SAN_DIR, exist_ok=True)
    objs = []
    for src in SOURCES:
        obj = os.path.join(SAN_DIR, src + ".o")
        if src in HOST_SOURCES:
            cmd = ["g++", "-std=c++17", "-fPIC", "-Wall", "-D__HIP_PLATFORM_AMD__", *SAN_FLAGS, "-I", INCLUDE,
                   "-I", CSRC, "-I", "/opt/rocm/include", "-c", os.path.join(CSRC, src), "-o", obj]
        else:
            cmd = [hipcc(), *HIP_FLAGS, "-I", INCLUDE, "-I", CSRC, "-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)
        objs.append(obj)
    # g++ links: the device code objects carry their own code-object sections
    cmd = ["g++", "-shared", "-fPIC", *SAN_FLAGS, *objs, "-o", SAN_LIB, "-L/opt/rocm/lib", "-lamdhip64",
           "-Wl,-rpath,/opt/rocm/lib"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    return SAN_LIB


def run_sanitized_tests(extra=()) -> int:
    """pytest -m "not gpu" with the sanitized copy loaded in place of the library."""
    runtimes = [subprocess.run(["g++", f"-print-file-name={n}"], capture_output=True, text=True, check=True)
                .stdout.strip() for n in ("libasan.so", "libubsan.so")]
    env = dict(os.environ)
    env["SF_DECODE_ATTN_LIB"] = SAN_LIB
    env["LD_PRELOAD"] = ":".join(runtimes)
    # Python itself is not instrumented: its allocations are not leaks of ours
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    cmd = [sys.executable, "-m", "pytest", os.path.join(ROOT, "tests"), "-q", "-m", "not gpu", *extra]
    return subprocess.run(cmd, env=env, cwd=ROOT).returncode


if __name__ == "__main__":
    if "--sanitize" in sys.argv:
        print(build_sanitized(verbose="-v" in sys.argv))
        if "--run-tests" in sys.argv:
            sys.exit(run_sanitized_tests())
    else:
        print(build(verbose="-v" in sys.argv))

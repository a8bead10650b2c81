"""Build of the HIP library (libforkstep.so) for gfx950.

``python -m paper_2609_39859_amd.build`` compiles the library's HIP sources
under csrc/ with hipcc into libforkstep.so next to this file, and the
benchmark's peak probes (csrc/peak_probe.hip) into libforkprobe.so.  The compile
disables packed-fp32 instruction selection (the -packed-fp32-ops target
feature); hipcc's host pass warns that it does not know the feature, which is
harmless.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libforkstep.so")
SOURCES = ["gemm_stats.hip", "merge_select.hip", "grpo.hip", "fork_abi.hip"]
PROBE_LIB = os.path.join(HERE, "libforkprobe.so")
PROBE_SOURCES = ["peak_probe.hip"]
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    return "hipcc"


def compile_flags():
    return ["-std=c++17", "-O3", "-fPIC", "--offload-arch=%s" % ARCH,
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-Wall", "-Wno-unused-result", "-I", INCLUDE, "-I", CSRC]


def build(verbose: bool = False) -> str:
    """Compile and link libforkstep.so and libforkprobe.so, then the plain-C
    example that drives one step through the C ABI; returns the path of
    libforkstep.so."""
    _build_lib(PROBE_LIB, PROBE_SOURCES, verbose)
    lib = _build_lib(LIB, SOURCES, verbose)
    build_c_example(verbose)
    return lib


C_EXAMPLE_SRC = os.path.join(ROOT, "tests", "native", "abi_c_step.c")
C_EXAMPLE = os.path.join(HERE, "_build", "abi_c_step")


def build_c_example(verbose: bool = False) -> str:
    """gcc -std=c99 build of tests/native/abi_c_step.c against the public
    header, libforkstep.so and the HIP runtime's C API."""
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    os.makedirs(os.path.dirname(C_EXAMPLE), exist_ok=True)
    cmd = ["gcc", "-std=c99", "-O1", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(rocm, "include"), "-I", INCLUDE, C_EXAMPLE_SRC,
           "-L", HERE, "-lforkstep", "-L", os.path.join(rocm, "lib"), "-lamdhip64", "-lm",
           "-Wl,-rpath,$ORIGIN/..", "-o", C_EXAMPLE]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    return C_EXAMPLE


def _build_lib(lib_path: str, sources, verbose: bool) -> str:
    objs = []
    builddir = os.path.join(HERE, "_build")
    os.makedirs(builddir, exist_ok=True)
    procs = []
    for src in sources:
        obj = os.path.join(builddir, os.path.splitext(src)[0] + ".o")
        cmd = [hipcc()] + compile_flags() + ["-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE,
                                            stderr=subprocess.STDOUT, text=True)))
        objs.append(obj)
    failed = []
    for src, p in procs:
        out, _ = p.communicate()
        # the host pass's note about the packed-fp32 feature is expected noise
        lines = [ln for ln in out.splitlines() if "packed-fp32-ops" not in ln]
        if lines and (verbose or p.returncode):
            print("\n".join(lines), file=sys.stderr)
        if p.returncode:
            failed.append(src)
    if failed:
        raise RuntimeError("hipcc failed for %s" % ", ".join(failed))
    tmp = lib_path + ".tmp%d" % os.getpid()
    cmd = [hipcc(), "-shared", "-fPIC", "--offload-arch=%s" % ARCH, "-o", tmp] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, lib_path)
    return lib_path


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))

"""Build libagft.so (HIP, gfx950) in-tree with hipcc."""
import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libagft.so")
SOURCES = [os.path.join(CSRC, "agft_step.hip"), os.path.join(CSRC, "agft_env.hip")]

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-Wall", "-Wno-unused-command-line-argument",
    # keep the compiler from emitting packed fp32 arithmetic
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def build(verbose=False, extra_flags=()):
    """Compile every HIP source into paper_2508_01744_amd/libagft.so."""
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    tmp = LIB + ".tmp"
    cmd = [hipcc, *HIPCC_FLAGS, *extra_flags, "-I", INCLUDE, *SOURCES, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


# the stream-ceiling measurement (bench.py), a library of its own
CEILING_SRC = os.path.join(CSRC, "stream_ceiling.hip")
CEILING_LIB = os.path.join(PKG, "libagft_ceiling.so")


def build_ceiling(verbose=False):
    """Compile the stream-ceiling kernels into paper_2508_01744_amd/libagft_ceiling.so."""
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    tmp = CEILING_LIB + ".tmp"
    cmd = [hipcc, *HIPCC_FLAGS, CEILING_SRC, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, CEILING_LIB)
    return CEILING_LIB


C_EXAMPLE_SRC = os.path.join(ROOT, "tests", "c_abi", "agft_c_example.c")
C_EXAMPLE = os.path.join(ROOT, "tests", "c_abi", "agft_c_example")


def build_c_example(verbose=False):
    """Compile the plain C caller of the ABI (host code, gcc) against libagft.so."""
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    cmd = ["gcc", "-std=c11", "-O2", "-Wall", "-D__HIP_PLATFORM_AMD__", "-I", INCLUDE,
           "-I", os.path.join(rocm, "include"), C_EXAMPLE_SRC, "-L", PKG, "-lagft",
           "-L", os.path.join(rocm, "lib"), "-lamdhip64",
           "-Wl,-rpath,$ORIGIN/../../paper_2508_01744_amd", "-Wl,-rpath," + os.path.join(rocm, "lib"),
           "-o", C_EXAMPLE]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    return C_EXAMPLE


if __name__ == "__main__":
    print(build(verbose=True))
    print(build_ceiling(verbose=True))

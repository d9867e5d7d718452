"""Build step for libwtconv.so (hipcc, gfx950), in-tree next to this file.

Every HIP source is compiled with packed-FP32 instructions disabled
(``-target-feature -packed-fp32-ops``); the kernels are written for plain
fp32 VALU FMAs.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libwtconv.so")
SOURCES = ["wtconv_api.cpp", "wtconv_kernels.hip", "wtconv_tiny.hip"]
# measurement helper used only by the benchmark (sustained VALU rate)
PROBE_LIB = os.path.join(HERE, "libvalu_probe.so")
PROBE_SOURCES = ["valu_probe.hip"]
ARCH = os.environ.get("WTCONV_OFFLOAD_ARCH", "gfx950")


def hipcc_flags():
    return ["--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-Wall",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-I", INCLUDE, "-I", CSRC]


def _compile(sources, lib, extra, verbose):
    hipcc = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")
    srcs = [os.path.join(CSRC, s) for s in sources]
    cmd = [hipcc] + hipcc_flags() + list(extra or []) + ["-shared", "-x", "hip"] + srcs + ["-o", lib + ".tmp"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(lib + ".tmp", lib)


def build(verbose: bool = False, extra=None) -> str:
    """Compile every HIP source (libwtconv.so and the benchmark's VALU probe)
    and return the path of libwtconv.so."""
    _compile(SOURCES, LIB, extra, verbose)
    _compile(PROBE_SOURCES, PROBE_LIB, extra, verbose)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))

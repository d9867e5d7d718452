"""Build step for libwtconv.so (hipcc, gfx950), in-tree next to this file.

Every HIP source is compiled with packed-FP32 instructions disabled
(``-target-feature -packed-fp32-ops``); the kernels are written for plain
fp32 VALU FMAs. Sources compile to objects in parallel (the forward and
backward instantiations of the fused kernel live in separate translation
units), then link into one shared library.
"""
import os
import subprocess
import tempfile
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libwtconv.so")
SOURCES = ["wtconv_api.cpp", "wtconv_noalloc.cpp", "wtconv_fwd.hip", "wtconv_mixed.hip", "wtconv_bwd.hip",
           "wtconv_bwd9.hip", "wtconv_grad.hip", "wtconv_kernels.hip", "wtconv_tiny.hip"]
# measurement helper used only by the benchmark (sustained VALU rate)
PROBE_LIB = os.path.join(HERE, "libvalu_probe.so")
PROBE_SOURCES = ["valu_probe.hip"]
ARCH = os.environ.get("WTCONV_OFFLOAD_ARCH", "gfx950")


def hipcc():
    return os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")


def hipcc_flags():
    return ["--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-Wall",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-I", INCLUDE, "-I", CSRC]


def _compile(sources, lib, extra, verbose):
    with tempfile.TemporaryDirectory(prefix="wtconv_build_") as tmp:
        def one(src):
            obj = os.path.join(tmp, src + ".o")
            cmd = [hipcc()] + hipcc_flags() + list(extra or []) + ["-x", "hip", "-c", os.path.join(CSRC, src),
                                                                    "-o", obj]
            if verbose:
                print(" ".join(cmd), flush=True)
            subprocess.run(cmd, check=True)
            return obj

        workers = max(1, min(len(sources), int(os.environ.get("MAX_JOBS", "8"))))
        with ThreadPoolExecutor(max_workers=workers) as pool:
            objs = list(pool.map(one, sources))
        cmd = [hipcc(), "--offload-arch=" + ARCH, "-shared", "-fPIC"] + objs + ["-o", lib + ".tmp"]
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

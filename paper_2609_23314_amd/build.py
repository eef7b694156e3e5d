"""Builds the HIP library ``libvd.so`` (kernels + C ABI) for gfx950 with hipcc,
and its debug build ``libvd_debug.so`` (VD_DEBUG=1: every dynamic LDS index
checked against the host's plan, see include/vd_debug.h).

    python -m paper_2609_23314_amd.build [-v] [--release-only]

The libraries are built in-tree, next to this file, so that they travel with
the source tree.  Every build compiles from scratch.
"""
import os
import shutil
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libvd.so")
DEBUG_LIB = os.path.join(HERE, "libvd_debug.so")
ARCH = "gfx950"

# Packed fp32 instructions are kept out of every device build.  MFMA results
# stay in ordinary VGPRs (the decode split kernel's accumulators would
# otherwise move to AGPRs and lower its occupancy).
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                "-mllvm", "-amdgpu-mfma-vgpr-form"]
COMMON = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-I", INCLUDE, "-I", CSRC]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    path = shutil.which("hipcc") or os.path.join(rocm, "bin", "hipcc")
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found; the HIP library cannot be built")
    return path


def _build_one(out: str, defines, verbose: bool) -> str:
    cc = hipcc()
    with tempfile.TemporaryDirectory() as tmp:
        objs = []
        steps = [
            [cc, f"--offload-arch={ARCH}", *COMMON, *defines, *DEVICE_FLAGS, "-c",
             os.path.join(CSRC, "vd_kernels.hip"), "-o", os.path.join(tmp, "vd_kernels.o")],
            [cc, *COMMON, *defines, "-x", "c++", "-D__HIP_PLATFORM_AMD__",
             "-I", os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "include"),
             "-c", os.path.join(CSRC, "vd_api.cpp"),
             "-o", os.path.join(tmp, "vd_api.o")],
        ]
        for cmd in steps:
            if verbose:
                print(" ".join(cmd), flush=True)
            subprocess.run(cmd, check=True)
            objs.append(cmd[-1])
        link = [cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", out + ".tmp", *objs]
        if verbose:
            print(" ".join(link), flush=True)
        subprocess.run(link, check=True)
    os.replace(out + ".tmp", out)
    return out


def build(verbose: bool = False, debug: bool = True) -> str:
    """Builds libvd.so and, unless debug is False, libvd_debug.so; returns the
    path of libvd.so."""
    _build_one(LIB, [], verbose)
    if debug:
        _build_one(DEBUG_LIB, ["-DVD_DEBUG=1"], verbose)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv, debug="--release-only" not in sys.argv))

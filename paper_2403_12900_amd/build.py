"""Builds the HIP decode library (libsprout.so, gfx950) and the host-only
bookkeeping test library (libsprout_host.so) in the package directory."""
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libsprout.so")
HOST_LIB = os.path.join(PKG, "libsprout_host.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
HIP_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # Packed fp32 instructions stay off: ordinary float code only.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # MFMA accumulators in VGPRs: epilogues and the softmax rescale operate on
    # them with VALU instructions, which cannot address AGPRs.
    "-mllvm", "-amdgpu-mfma-vgpr-form",
    # The leading scalar kernel arguments (pointers, sizes) arrive preloaded in
    # SGPRs, so a kernel's first loads need not wait for its argument fetch.
    "-mllvm", "-amdgpu-kernarg-preload-count=16",
    "-Wno-unused-result",
]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)


def build(verbose: bool = True) -> None:
    srcs = [os.path.join(CSRC, "sprout.hip"), os.path.join(CSRC, "host_state.cpp")]
    tmp = LIB + ".tmp"
    _run([HIPCC, *HIP_FLAGS, *srcs, "-o", tmp], verbose)
    os.replace(tmp, LIB)
    tmp = HOST_LIB + ".tmp"
    _run(["g++", "-O2", "-std=c++17", "-fPIC", "-shared", "-Wall",
          os.path.join(CSRC, "host_state.cpp"), os.path.join(CSRC, "host_test_api.cpp"), "-o", tmp], verbose)
    os.replace(tmp, HOST_LIB)


if __name__ == "__main__":
    build(verbose="-q" not in sys.argv)

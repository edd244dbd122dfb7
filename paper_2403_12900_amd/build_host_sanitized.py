"""Builds the host-only bookkeeping library (slot table, KV-block pool, scheduler) a second time with
AddressSanitizer and UndefinedBehaviorSanitizer, for the CPU tests: libsprout_host_asan.so in the
package directory.  Host code only; no device code is built here."""
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
ASAN_LIB = os.path.join(PKG, "libsprout_host_asan.so")
SANITIZE = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer"]


def build(verbose: bool = True) -> str:
    tmp = ASAN_LIB + ".tmp"
    cmd = ["g++", "-O1", "-g", "-std=c++17", "-fPIC", "-shared", "-Wall", *SANITIZE,
           os.path.join(CSRC, "host_state.cpp"), os.path.join(CSRC, "host_test_api.cpp"), "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, ASAN_LIB)
    return ASAN_LIB


def runtime_preload() -> str:
    """The sanitizer runtimes a non-instrumented Python must preload to load the library."""
    libs = []
    for name in ("libasan.so", "libubsan.so"):
        p = subprocess.run(["g++", f"-print-file-name={name}"], capture_output=True, text=True, check=True).stdout.strip()
        libs.append(os.path.realpath(p))
    return ":".join(libs)


if __name__ == "__main__":
    build(verbose="-q" not in sys.argv)

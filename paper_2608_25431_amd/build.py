"""Builds the HIP library libgift.so (gfx950) in-tree, and libgift_probe.so
(LDS-rate probes for the benchmark).

    python -m paper_2608_25431_amd.build
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libgift.so")
SOURCES = [os.path.join(CSRC, "gift_kernels.hip"), os.path.join(CSRC, "gift_host.cpp"), os.path.join(CSRC, "gift_ift.cpp")]
PROBE_SOURCE = os.path.join(CSRC, "gift_probe.hip")
PROBE_LIB = os.path.join(HERE, "libgift_probe.so")
ARCH = "gfx950"

# Packed-FP32 instructions are disabled for all device code.
HIP_FLAGS = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _hipcc(sources, lib, verbose):
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    tmp = lib + ".tmp"
    cmd = [hipcc, f"--offload-arch={ARCH}", *HIP_FLAGS, "-shared", "-I", os.path.join(ROOT, "include"),
           "-I", CSRC, *sources, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass reports the device-only target feature as unknown: harmless
    noise = [l for l in r.stderr.splitlines() if l.strip() and "packed-fp32-ops" not in l]
    if r.returncode != 0:
        sys.stderr.write(r.stderr)
        raise RuntimeError(f"hipcc failed ({r.returncode})")
    if verbose and noise:
        sys.stderr.write("\n".join(noise) + "\n")
    os.replace(tmp, lib)


def build(verbose: bool = False) -> str:
    """The library, and the LDS-rate probes the benchmark loads beside it."""
    _hipcc(SOURCES, LIB, verbose)
    _hipcc([PROBE_SOURCE], PROBE_LIB, verbose)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))

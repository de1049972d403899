"""Builds the two workload-generator libraries in place.

libbaton_wl_host.so (gcc, OpenMP) and libbaton_wl_dev.so (hipcc, gfx950) are
compiled from the same value function in csrc/wl_core.h.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
HOST_LIB = os.path.join(HERE, "libbaton_wl_host.so")
DEV_LIB = os.path.join(HERE, "libbaton_wl_dev.so")

HIP_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", "-shared", "--offload-arch=gfx950",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def _run(cmd):
    subprocess.run(cmd, check=True, cwd=HERE)


def build(verbose=False):
    src = os.path.join(HERE, "csrc")
    host = ["gcc", "-O3", "-std=c11", "-fPIC", "-shared", "-fopenmp",
            os.path.join(src, "wl_host.c"), "-o", HOST_LIB + ".tmp"]
    dev = ["hipcc", *HIP_FLAGS, os.path.join(src, "wl_device.hip"), "-o", DEV_LIB + ".tmp"]
    for cmd, out in ((host, HOST_LIB), (dev, DEV_LIB)):
        if verbose:
            print(" ".join(cmd), flush=True)
        _run(cmd)
        os.replace(out + ".tmp", out)


if __name__ == "__main__":
    build(verbose=True)

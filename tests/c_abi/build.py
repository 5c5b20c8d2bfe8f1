"""Builds abi_check (abi_check.cpp, a host program that uses the C ABI with
plain device pointers) next to its source, linked against the in-tree
libdg.so (found at run time through an rpath relative to the program)."""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
PKG = os.path.join(ROOT, "paper_2405_05231_amd")
EXE = os.path.join(HERE, "abi_check")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def build(verbose: bool = False) -> str:
    tmp = EXE + ".tmp"
    cmd = [HIPCC, "-O2", "-std=c++17", "--offload-arch=gfx950", "-Wall",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I", os.path.join(ROOT, "include"), os.path.join(HERE, "abi_check.cpp"),
           "-L", PKG, "-ldg", "-Wl,-rpath,$ORIGIN/../../paper_2405_05231_amd", "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, EXE)
    return EXE


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))

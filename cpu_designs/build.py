"""Compile the paper's CPU designs into cpu_designs/libcpudesigns.so (g++ with
OpenMP; FP contraction off, so that every FP32 add and multiply rounds as the
paper's loops write them)."""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "designs.cpp")
LIB = os.path.join(HERE, "libcpudesigns.so")
FLAGS = ["-O3", "-std=c++17", "-fopenmp", "-fno-fast-math", "-ffp-contract=off", "-shared",
         "-fPIC"]


def build(verbose: bool = False) -> str:
    tmp = LIB + f".tmp{os.getpid()}"
    cmd = ["g++", *FLAGS, SRC, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))

"""Build the CPU oracle library (oracle/liboracle.so) with g++.

Test infrastructure: the product library never links or loads it.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "moe_oracle.cpp")
LIB = os.path.join(HERE, "liboracle.so")

# -ffp-contract=off: every multiply and add rounds on its own (no fused
# multiply-add), as the oracle's arithmetic is written.
CMD = ["g++", "-O2", "-std=c++17", "-ffp-contract=off", "-fno-fast-math",
       "-Wall", "-Wextra", "-shared", "-fPIC", SRC, "-o", LIB]


def build(verbose: bool = False) -> str:
    if verbose:
        print(" ".join(CMD), flush=True)
    subprocess.run(CMD, check=True)
    return LIB


if __name__ == "__main__":
    build(verbose=True)

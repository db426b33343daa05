"""Compile the float64 oracle (plain C, gcc) into oracle/liblocaoracle.so.

Test infrastructure: the product path never loads this library.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "loca_oracle.c")
LIB = os.path.join(HERE, "liblocaoracle.so")


def build_oracle(verbose: bool = False) -> str:
    # Portable x86-64 code (the library travels to other hosts); no fast-math.
    cmd = ["gcc", "-O2", "-std=c99", "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra",
           "-o", LIB + ".tmp", SRC, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.check_call(cmd)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    print(build_oracle(verbose=True))

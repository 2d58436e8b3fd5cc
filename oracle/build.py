"""Compile the fp64 CPU oracles of the MoE layer and the attention block (test
infrastructure) into oracle/libmoe_oracle.so.

Plain C11 built with gcc, OpenMP over output columns and tokens; no
-ffast-math, so every sum keeps its written order.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRCS = [os.path.join(HERE, "moe_oracle.c"), os.path.join(HERE, "attn_oracle.c")]
LIB = os.path.join(HERE, "libmoe_oracle.so")


def build(force: bool = True) -> str:
    if (not force and os.path.exists(LIB) and
            os.path.getmtime(LIB) >= max(os.path.getmtime(s) for s in SRCS)):
        return LIB
    tmp = LIB + ".tmp"
    cmd = ["gcc", "-std=c11", "-O2", "-fno-fast-math", "-ffp-contract=off", "-fopenmp",
           "-fPIC", "-shared", "-Wall", "-Wextra", "-o", tmp] + SRCS + ["-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build())

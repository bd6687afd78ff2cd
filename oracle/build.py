"""Build the CPU oracle library (plain C, double precision, OpenMP).

TEST INFRASTRUCTURE ONLY: the oracle checks and times the HIP path; the
product path never builds, loads or calls it.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRCS = [os.path.join(HERE, "pa_oracle.c"), os.path.join(HERE, "pa_oracle_block.c")]
LIB = os.path.join(HERE, "libpa_oracle.so")


def build(verbose: bool = False) -> str:
    """Compile the oracle's C sources into oracle/libpa_oracle.so and return its path.

    Portable flags only (no -march=native): the library is built here and
    also loaded on other hosts.
    """
    tmp = LIB + ".tmp"
    cmd = ["gcc", "-std=c11", "-O2", "-fopenmp", "-fPIC", "-shared",
           "-Wall", "-Wextra", "-o", tmp, *SRCS, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))

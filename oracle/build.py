"""Build the CPU oracle library (plain C, double precision, OpenMP).

TEST INFRASTRUCTURE ONLY: the oracle checks and times the HIP path; the
product path never builds, loads or calls it.

Variants (one library file each):
  portable   -O2, no host-specific instructions: built here and loaded on
             other hosts too (the default)
  native     -O3 -march=native: built on the host that then times it (the
             CPU baseline of the benchmark), never shipped to another host
  sanitized  AddressSanitizer + UndefinedBehaviorSanitizer, every UB report
             fatal: the oracle's pins are also run against it
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRCS = [os.path.join(HERE, "pa_oracle.c"), os.path.join(HERE, "pa_oracle_block.c")]
LIB = os.path.join(HERE, "libpa_oracle.so")
VARIANTS = {
    "portable": (LIB, ["-O2"]),
    "native": (os.path.join(HERE, "libpa_oracle_native.so"), ["-O3", "-march=native"]),
    "sanitized": (os.path.join(HERE, "libpa_oracle_san.so"),
                  ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                   "-fno-sanitize-recover=undefined"]),
}


def lib_path(variant: str = "portable") -> str:
    return VARIANTS[variant][0]


def build(verbose: bool = False, variant: str = "portable") -> str:
    """Compile the oracle's C sources into the variant's library and return its path."""
    out, flags = VARIANTS[variant]
    tmp = out + ".tmp"
    cmd = ["gcc", "-std=c11", *flags, "-fopenmp", "-fPIC", "-shared",
           "-Wall", "-Wextra", "-o", tmp, *SRCS, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))

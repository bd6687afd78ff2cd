"""Build the gfx950 HIP library ``libpa.so`` in-tree with hipcc.

Every source under ``csrc/`` is compiled for gfx950 only, in parallel, and
linked into ``paper_2502_02414_amd/libpa.so`` (the C ABI of include/pa.h).
"""
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libpa.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SOURCES = ["pa_stream.hip", "pa_stream_agg.hip", "pa_stream_des.hip", "pa_stream_desbwd.hip",
           "pa_stream_wts.hip", "pa_stream_slbwd.hip", "pa_stream_wtsbwd.hip", "pa_small.hip",
           "pa_stream_aggw.hip", "pa_stream_desw.hip", "pa_stream_desbwdw.hip", "pa_tokens.hip",
           "pa_tokens64.hip", "pa_block.hip", "pa_mlp.hip", "pa_heads.hip", "pa_probe.hip", "pa_api.cpp", "pa_gemm.cpp", "pa_block_api.cpp"]
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-fPIC", "-std=c++17",
    # packed-FP32 VALU forms are kept out of the device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function", "-Wno-unused-variable",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
]


def _compile(src: str, verbose: bool) -> str:
    obj = os.path.join(OUT, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, "-x", "hip", *FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = False) -> str:
    """Compile every source and link libpa.so; returns the library path."""
    os.makedirs(OUT, exist_ok=True)
    with ThreadPoolExecutor(min(len(SOURCES), os.cpu_count() or 4)) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), SOURCES))
    tmp = LIB + ".tmp"
    # hipBLASLt for the block stack's plain GEMMs
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs,
           "-L/opt/rocm/lib", "-lhipblaslt"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))

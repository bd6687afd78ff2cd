"""Benchmark: one Physics-Attention layer, forward + backward, on one MI355X.

A step is one pass of the whole hot path over one batch of synthetic input:
    pa_slice_aggregate -> pa_token_attention -> pa_deslice        (forward)
    pa_deslice_backward -> pa_token_attention_backward
                        -> pa_slice_aggregate_backward           (backward)
on the million-point car-surface workload (N = 1,000,000, C = 256, H = 8,
M = 32, bf16 storage, fp32 accumulation).  Inputs are resident in HBM before
the timed region.  Prints one JSON line (rank 0).  The headline is this
sequence, which recomputes the slice weights in every pass; the line also
reports, under "stored_weights", the same step with the weights written once
by pa_slice_aggregate_w and read by pa_deslice_w / pa_deslice_backward_w.

    python bench.py [--gpus 1] [--steps 20] [--warmup 3] [--no-cpu-baseline]

Roofline: the streaming kernel of the dominant call is timed with HIP events
over every timed step: the library records them on the stream it launches on,
right around that kernel (pa_time_kernel), so the duration is the kernel's
own, as rocprofv3 reports it.  Its achieved bandwidth is its algorithmic
bytes per launch over that duration.  Traffic (HBM
bytes per call from the rocprofv3 FETCH_SIZE / WRITE_SIZE counters) is read
from profiles/traffic_*.txt when that file was measured on the current
kernel sources, else null.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = ("mesh points/sec per Physics-Attention layer fwd+bwd at N=1M, C=256, M=32; "
          "% roofline")
WORKLOAD = "car_1m_bf16"
HBM_PEAK_GBS = 8000.0
# Algorithmic HBM bytes per point of each streaming call (b = 2, g = 2 for
# bf16): the inputs each call must read and the outputs it must write.
def algo_bytes_per_point(C, M, b, g):
    return {
        "pa_slice_aggregate": C * b + M * g,           # x, G
        "pa_deslice": 2 * C * b + M * g,               # x, G, y
        "pa_deslice_backward": 2 * C * b + M * g,      # x, G, dY
        "pa_slice_aggregate_backward": 3 * C * b + M * g,  # x, G, dY, dx
        "pa_token_attention": 0,
        "pa_token_attention_backward": 0,
        # stored weights: W [N,M] written once, read in place of x and G
        "pa_slice_aggregate_w": C * b + M * g + M * b,   # x, G read; W written
        "pa_deslice_w": M * b + C * b,                  # W read; y written
        "pa_deslice_backward_w": M * b + C * b,         # W, dY read
    }


# Algorithmic MFMA flops per point of each streaming call: the logits
# contraction (2 C M) plus the call's own contraction over C and M (2 C M);
# the slice backward has the logits, dw from the deslice term dY S'^T and
# from the states term x dnum^T, dx = dl A^T + W dnum and dA = x^T dl
# (12 C M in all); the stored-weights deslice and its backward only their
# own contraction.
def algo_flops_per_point(C, M):
    return {"pa_slice_aggregate": 4 * C * M, "pa_deslice": 4 * C * M,
            "pa_deslice_backward": 4 * C * M, "pa_slice_aggregate_backward": 12 * C * M,
            "pa_slice_aggregate_w": 4 * C * M, "pa_deslice_w": 2 * C * M,
            "pa_deslice_backward_w": 2 * C * M}


MFMA_PEAK_TFLOPS = 2500.0   # dense bf16


# The streaming kernel each call launches (one per call).
STREAM_KERNEL = {
    "pa_slice_aggregate": "aggregate",          # k_aggregate, forward
    "pa_deslice": "deslice",                    # k_deslice
    "pa_deslice_backward": "deslice_bwd",       # k_aggregate, deslice backward
    "pa_slice_aggregate_backward": "slice_bwd",  # k_slice_bwd
    "pa_slice_aggregate_w": "aggregate_w",
    "pa_deslice_w": "deslice_w",
    "pa_deslice_backward_w": "deslice_bwd_w",
}


# The sources the streaming kernels are compiled from (the traffic summary
# is valid while these are unchanged).
STREAM_SOURCES = ("pa_device.hpp", "pa_internal.h", "pa_layout.h", "pa_stream.hpp",
                  "pa_stream_slbwd.hip", "pa_coop.hpp")


def kernel_sources_sha() -> str:
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2502_02414_amd", "csrc")
    for name in STREAM_SOURCES:
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(name.encode())
            h.update(f.read())
    return h.hexdigest()[:16]


def read_traffic(kernel: str):
    """Per-call HBM bytes (fetch + write) measured by rocprofv3 counters, if the
    summary in profiles/ was taken on the current kernel sources."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{WORKLOAD}.txt")
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                vals[k.strip()] = v.strip()
    if vals.get("kernel_sources_sha") != kernel_sources_sha():
        return None
    try:
        return float(vals["hbm_bytes_per_call"])
    except (KeyError, ValueError):
        return None


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain 1 GiB device copy (counter calibration)")
    ap.add_argument("--stack", action="store_true",
                    help="time the 8-block Transolver++ stack at N = 2.5M instead (its own line)")
    ap.add_argument("--heads", action="store_true",
                    help="time the per-head sliced layer at N = 1M instead (its own line)")
    ap.add_argument("--head-streams", type=int, default=2,
                    help="streams the per-head layer spreads its heads over (one call per head)")
    ap.add_argument("--workload", default=None,
                    help="time the layer on another workload instead (its own line): "
                         "ns2d_fwd_f32, grid2d_16k_f32, ellipsoid_32k_bf16, aircraft_2p5m_bf16")
    ap.add_argument("--flush", action="store_true",
                    help="with --workload: overwrite 1 GiB between steps (cold last-level cache)")
    ap.add_argument("--probe", action="store_true",
                    help="time each streaming kernel of the layer (in the step) beside a probe "
                         "moving the same tensors the same way with no arithmetic "
                         "(pa_stream_probe); the headline workload unless --workload")
    ap.add_argument("--graph", action="store_true",
                    help="with --workload: replay the step from a captured HIP graph")
    ap.add_argument("--head-calls", choices=("batched", "per-head"), default=None,
                    help="per-head layer: all heads in one launch per kernel, or one call per head")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the library runs the "
              "hot path on a single MI355X and has no multi-GPU path.", file=sys.stderr)
        sys.exit(2)
    if args.stack:
        return stack_bench(args)
    if args.heads:
        return heads_bench(args)
    if args.probe:
        args.workload = args.workload or WORKLOAD
        return workload_bench(args)
    if args.workload:
        return workload_bench(args)

    import numpy as np
    import torch
    from paper_2502_02414_amd import binding as B
    from paper_2502_02414_amd import inputs as I

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = I.WORKLOADS[WORKLOAD]
    N, C, H, M = w.N, w.C, w.H, w.M

    t0 = time.time()
    x_np = I.make_x(w)
    G_np = I.make_gumbel(w)
    dY_np = I.make_grad(w)
    p = I.make_params(w)
    print(f"[bench] inputs generated in {time.time() - t0:.1f}s", file=sys.stderr, flush=True)

    bf = torch.bfloat16
    to = lambda a, dt=torch.float32: torch.from_numpy(np.ascontiguousarray(a)).to(dev).to(dt)
    x, G, dY = to(x_np, bf), to(G_np, bf), to(dY_np, bf)
    A, a = to(p["A"], bf), to(p["a"], bf)
    b = to(p["b"])
    att = {k: to(p[k]) for k in ("Wq", "bq", "Wk", "bk", "Wv", "bv")}
    dims = B.make_dims(N, C, H, M, w.tau0, w.tau_min, w.eps, B.PA_BF16)
    sp = B.make_slice_params(A, b, a, p["b_t"])
    apr = B.make_attn_params(**att)
    ws = B.workspace(dims, dev)
    f32 = lambda *s: torch.empty(*s, dtype=torch.float32, device=dev)
    num, den, S, Sp, dSp, dS = f32(M, C), f32(M), f32(M, C), f32(M, C), f32(M, C), f32(M, C)
    y = torch.empty(N, C, dtype=bf, device=dev)
    dx = torch.empty(N, C, dtype=bf, device=dev)
    ag = {k: f32(C, C) for k in ("dWq", "dWk", "dWv")}
    ag.update({k: f32(C) for k in ("dbq", "dbk", "dbv")})
    agr = B.make_attn_grads(**ag)
    sg = {"dA": f32(C, M), "db": f32(M), "da": f32(C), "db_t": f32(1), "dtau0": f32(1)}
    sgr = B.make_slice_grads(**sg)

    calls = [
        ("pa_slice_aggregate", lambda: B.pa_slice_aggregate(dims, x, G, sp, num, den, S, ws)),
        ("pa_token_attention", lambda: B.pa_token_attention(dims, S, apr, Sp, ws)),
        ("pa_deslice", lambda: B.pa_deslice(dims, x, G, sp, Sp, y, ws)),
        ("pa_deslice_backward", lambda: B.pa_deslice_backward(dims, x, G, sp, dY, dSp, ws)),
        ("pa_token_attention_backward",
         lambda: B.pa_token_attention_backward(dims, S, apr, dSp, dS, agr, ws)),
        ("pa_slice_aggregate_backward",
         lambda: B.pa_slice_aggregate_backward(dims, x, G, sp, num, den, dS, Sp, dY, dx, sgr, ws)),
    ]

    Wst = torch.empty(N, M, dtype=bf, device=dev)  # stored weights (variant)
    calls_w = [
        ("pa_slice_aggregate_w",
         lambda: B.pa_slice_aggregate_w(dims, x, G, sp, num, den, S, Wst, ws)),
        calls[1],
        ("pa_deslice_w", lambda: B.pa_deslice_w(dims, Wst, Sp, y, ws)),
        ("pa_deslice_backward_w", lambda: B.pa_deslice_backward_w(dims, Wst, dY, dSp, ws)),
        calls[4],
        calls[5],
    ]

    bpp = algo_bytes_per_point(C, M, 2, 2)
    headline = time_steps(calls, bpp, args, B, torch)
    variant = time_steps(calls_w, bpp, args, B, torch)
    dom, per_call, kernel_ms = headline["dom"], headline["per_call"], headline["kernel_ms"]
    ms_per_step, t_wall = headline["ms_per_step"], headline["wall_s"]
    value = N / (ms_per_step * 1e-3)

    if args.copy_calibration:
        src = torch.empty(1 << 28, dtype=torch.float32, device=dev)  # 1 GiB
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    dom_bytes = bpp[dom] * N
    achieved = dom_bytes / (kernel_ms * 1e-3) / 1e9
    step_bytes = sum(bpp[n] for n, _ in calls) * N
    w_bytes = sum(bpp[n] for n, _ in calls_w) * N
    w_ms = variant["ms_per_step"]
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                "traffic": read_traffic(STREAM_KERNEL[dom]), "call": dom,
                "kernel": STREAM_KERNEL[dom], "algo_bytes_per_launch": dom_bytes,
                "kernel_ms": round(kernel_ms, 4), "call_ms": round(per_call[dom], 4)}
    # the same kernel against the dense bf16 MFMA peak (it is HBM-bound)
    dom_flops = algo_flops_per_point(C, M)[dom] * N
    tflops = dom_flops / (kernel_ms * 1e-3) / 1e12
    mfma = {"achieved": round(tflops, 1), "peak": MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": round(tflops / MFMA_PEAK_TFLOPS, 4), "algo_flops_per_launch": dom_flops}

    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "points/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": WORKLOAD, "N": N, "C": C, "H": H, "M": M, "tau0": w.tau0,
                   "tau_min": w.tau_min, "storage": "bf16", "accumulate": "fp32",
                   "pass": "forward+backward"},
        "roofline": roofline,
        "mfma": mfma,
        "step_hbm": {"algo_bytes": step_bytes,
                     "achieved_GBs": round(step_bytes / (ms_per_step * 1e-3) / 1e9, 1),
                     "frac": round(step_bytes / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)},
        "per_call_ms": {k: round(v, 4) for k, v in per_call.items()},
        "wall_s_timed": round(t_wall, 4),
        # Algorithm 1's dataflow: the weights stored once by the aggregate and
        # read by the deslice and its backward (same workload and outputs)
        "stored_weights": {
            "value": round(N / (w_ms * 1e-3), 1), "ms_per_step": round(w_ms, 4),
            "algo_bytes": w_bytes,
            "achieved_GBs": round(w_bytes / (w_ms * 1e-3) / 1e9, 1),
            "frac": round(w_bytes / (w_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "per_call_ms": {k: round(v, 4) for k, v in variant["per_call"].items()}},
    }

    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(x_np, G_np, dY_np, p, w,
                                           per_core=I.WORKLOADS["ellipsoid_32k_bf16"])
    print(json.dumps(out), flush=True)


def probe_report(args, w, dims, step, x, G, dY, out, B, torch):
    """Each streaming kernel timed inside the layer's step (pa_time_kernel,
    median of the steps) beside pa_stream_probe for the same call: the same
    tensors moved by the same blocks, waves, tiles, prefetch, walk direction
    and cache hints, with no arithmetic (median of as many probes, each after
    a 1 GiB write so that no input is left in the last-level cache; inside
    the step a kernel may find part of its input there).  Prints one JSON
    line."""
    N, C, M = w.N, w.C, w.M
    sz = 2 if w.dtype == "bf16" else 4
    bpp = algo_bytes_per_point(C, M, sz, sz)
    calls = ["pa_slice_aggregate", "pa_deslice"] + (
        ["pa_deslice_backward", "pa_slice_aggregate_backward"] if w.backward else [])
    reps = max(3, args.steps)
    junk = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
    e0, e1 = B.HipEvent(), B.HipEvent()
    passes = {}
    for c in calls:
        B.pa_time_kernel(c, e0, e1)
        kt = []
        for _ in range(reps):
            step()
            torch.cuda.synchronize()
            kt.append(e0.elapsed_ms(e1))
        B.pa_time_kernel(None)
        reads_dy = c in ("pa_deslice_backward", "pa_slice_aggregate_backward")
        writes = c in ("pa_deslice", "pa_slice_aggregate_backward")
        pt = []
        for r in range(reps):
            junk.fill_(float(r))
            e0.record()
            B.pa_stream_probe(dims, c, x, dY if reads_dy else None, G, out if writes else None)
            e1.record()
            torch.cuda.synchronize()
            pt.append(e0.elapsed_ms(e1))
        k_ms, p_ms = sorted(kt)[len(kt) // 2], sorted(pt)[len(pt) // 2]
        nb = bpp[c] * N
        passes[c] = {"kernel": STREAM_KERNEL[c], "algo_bytes": nb,
                     "kernel_us": round(k_ms * 1e3, 1), "probe_us": round(p_ms * 1e3, 1),
                     "kernel_GBs": round(nb / (k_ms * 1e-3) / 1e9, 1),
                     "probe_GBs": round(nb / (p_ms * 1e-3) / 1e9, 1),
                     "kernel_over_probe": round(p_ms / k_ms, 4)}
    out_line = {"probe": w.name, "N": N, "C": C, "M": M, "dtype": w.dtype, "reps": reps,
                "kernel_sources_sha": kernel_sources_sha(), "peak_GBs": HBM_PEAK_GBS,
                "passes": passes}
    print(json.dumps(out_line), flush=True)


def stack_bench(args):
    """The 8-block Transolver++ stack (LN -> Physics-Attention with the folded
    Project step -> MLP 256-1024-256 with GELU, residual adds) at N = 2.5M
    points, C = 256, H = 8, M = 64, bf16, forward + backward on one GPU: one
    step is the stack's forward and backward (no optimizer step).  Prints its
    own JSON line; the headline line is the layer's."""
    import torch
    from paper_2502_02414_amd import binding as B
    from paper_2502_02414_amd import inputs as I
    from paper_2502_02414_amd.stack import BlockStack

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    w = I.WORKLOADS["aircraft_2p5m_bf16"]
    N, C, H, M, L = w.N, w.C, w.H, w.M, 8
    t0 = time.time()
    bf = torch.bfloat16
    to = lambda a, dt=torch.float32: torch.from_numpy(a).cuda().to(dt)
    x, dY = to(I.make_x(w), bf), to(I.make_grad(w), bf)
    Gs = [to(I.make_layer_gumbel(w, l), bf) for l in range(L)]
    params = []
    for l in range(L):
        p = I.make_block_params(w, l)
        params.append({k: (float(v) if k == "b_t" else to(v, bf if k in ("W1", "W2") else
                                                         torch.float32)) for k, v in p.items()})
    print(f"[bench] stack inputs generated in {time.time() - t0:.1f}s", file=sys.stderr,
          flush=True)
    st = BlockStack(N, C, H, M, params, bf, w.tau0, w.tau_min, w.eps)
    steps, warmup = max(1, min(args.steps, 5)), max(1, min(args.warmup, 2))
    ev = [[B.HipEvent() for _ in range(3)] for _ in range(steps)]
    for _ in range(warmup):
        st.forward(x, Gs)
        st.backward(dY)
    torch.cuda.synchronize()
    start, end = B.HipEvent(), B.HipEvent()
    start.record()
    for s in range(steps):
        ev[s][0].record()
        st.forward(x, Gs)
        ev[s][1].record()
        st.backward(dY)
        ev[s][2].record()
    end.record()
    torch.cuda.synchronize()
    ms = start.elapsed_ms(end) / steps
    fwd = sum(e[0].elapsed_ms(e[1]) for e in ev) / steps
    bwd = sum(e[1].elapsed_ms(e[2]) for e in ev) / steps
    # MLP GEMM flops per step: forward 2 GEMMs, backward 4, each 2 N C 4C
    mlp_flop = 6 * 2 * N * C * 4 * C * L
    out = {
        "metric": "mesh points/sec, 8-block Transolver++ stack fwd+bwd at N=2.5M, C=256, M=64",
        "value": round(N / (ms * 1e-3), 1), "unit": "points/s", "n_gpus": 1, "steps": steps,
        "warmup": warmup, "ms_per_step": round(ms, 2), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "aircraft_2p5m_bf16_8blocks", "N": N, "C": C, "H": H, "M": M,
                   "blocks": L, "mlp_hidden": 4 * C, "pass": "forward+backward"},
        "forward_ms": round(fwd, 2), "backward_ms": round(bwd, 2),
        "mlp_gemm_tflops": round(mlp_flop / (ms * 1e-3) / 1e12, 1),
        "peak_mem_gib": round(torch.cuda.max_memory_allocated() / 2**30, 1),
    }
    print(json.dumps(out), flush=True)


def workload_bench(args):
    """The layer's call sequence on another workload (forward only when the
    workload is), each step bracketed by its own events; with --flush a
    1 GiB buffer is overwritten before every step (outside the events), so
    that no input is left in the 256 MB last-level cache.  Prints its own
    JSON line (the headline line is the million-point one)."""
    import numpy as np
    import torch
    from paper_2502_02414_amd import binding as B
    from paper_2502_02414_amd import inputs as I

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    w = I.WORKLOADS[args.workload]
    N, C, H, M = w.N, w.C, w.H, w.M
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    pdt = B.PA_BF16 if w.dtype == "bf16" else B.PA_F32
    to = lambda a, t=torch.float32: torch.from_numpy(np.ascontiguousarray(a)).cuda().to(t)
    p = I.make_params(w)
    x, G, dY = to(I.make_x(w), dt), to(I.make_gumbel(w), dt), to(I.make_grad(w), dt)
    A, a, b = to(p["A"], dt), to(p["a"], dt), to(p["b"])
    att = {k: to(p[k]) for k in ("Wq", "bq", "Wk", "bk", "Wv", "bv")}
    dims = B.make_dims(N, C, H, M, w.tau0, w.tau_min, w.eps, pdt)
    sp, apr, ws = B.make_slice_params(A, b, a, p["b_t"]), B.make_attn_params(**att), B.workspace(dims)
    f32 = lambda *s: torch.empty(*s, dtype=torch.float32, device="cuda")
    num, den, S, Sp, dSp, dS = f32(M, C), f32(M), f32(M, C), f32(M, C), f32(M, C), f32(M, C)
    y, dx = torch.empty(N, C, dtype=dt, device="cuda"), torch.empty(N, C, dtype=dt, device="cuda")
    ag = {k: f32(C, C) for k in ("dWq", "dWk", "dWv")}
    ag.update({k: f32(C) for k in ("dbq", "dbk", "dbv")})
    agr = B.make_attn_grads(**ag)
    sgr = B.make_slice_grads(dA=f32(C, M), db=f32(M), da=f32(C), db_t=f32(1), dtau0=f32(1))

    def step():
        B.pa_slice_aggregate(dims, x, G, sp, num, den, S, ws)
        B.pa_token_attention(dims, S, apr, Sp, ws)
        B.pa_deslice(dims, x, G, sp, Sp, y, ws)
        if w.backward:
            B.pa_deslice_backward(dims, x, G, sp, dY, dSp, ws)
            B.pa_token_attention_backward(dims, S, apr, dSp, dS, agr, ws)
            B.pa_slice_aggregate_backward(dims, x, G, sp, num, den, dS, Sp, dY, dx, sgr, ws)

    junk = torch.empty(1 << 28, dtype=torch.float32, device="cuda") if args.flush else None
    for _ in range(args.warmup):
        step()
    if args.probe:
        return probe_report(args, w, dims, step, x, G, dY, y, B, torch)
    if args.graph:
        # capture the step once on a side stream, then time its replays (the
        # library's calls only launch kernels: capturable as they are)
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step()
        torch.cuda.current_stream().wait_stream(side)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        step = graph.replay
        step()
    ev = [(B.HipEvent(), B.HipEvent()) for _ in range(args.steps)]
    torch.cuda.synchronize()
    for e0, e1 in ev:
        if junk is not None:
            junk.fill_(1.0)
        e0.record()
        step()
        e1.record()
    torch.cuda.synchronize()
    times = sorted(e0.elapsed_ms(e1) for e0, e1 in ev)
    ms = times[len(times) // 2]
    if args.copy_calibration:  # a 1 GiB copy for the HBM counters' scale, after the timing
        src = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    bpp = algo_bytes_per_point(C, M, 2 if w.dtype == "bf16" else 4, 2 if w.dtype == "bf16" else 4)
    calls = ["pa_slice_aggregate", "pa_deslice"] + (
        ["pa_deslice_backward", "pa_slice_aggregate_backward"] if w.backward else [])
    nbytes = N * sum(bpp[c] for c in calls)
    gbs = nbytes / (ms * 1e-3) / 1e9
    out = {
        "metric": f"mesh points/sec per Physics-Attention layer "
                  f"{'fwd+bwd' if w.backward else 'fwd'} at N={N}, C={C}, M={M}",
        "value": round(N / (ms * 1e-3), 1), "unit": "points/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "ms_per_step_min": round(times[0], 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": w.name, "N": N, "C": C, "H": H, "M": M,
                   "pass": "forward+backward" if w.backward else "forward",
                   "cache": "flushed before every step" if args.flush else "warm",
                   "launch": "HIP graph replay" if args.graph else "eager"},
        "step_hbm": {"algo_bytes": nbytes, "achieved_GBs": round(gbs, 1),
                     "frac": round(gbs / HBM_PEAK_GBS, 4)},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(I.make_x(w), I.make_gumbel(w), I.make_grad(w), p, w)
    print(json.dumps(out), flush=True)


def heads_bench(args):
    """Per-head slicing at the million-point car workload's shape: N = 1M,
    C = 256 as H = 8 heads of D = 32 channels, M = 32 slices per head (each
    head its own slice parameters and noise), bf16, forward + backward on the
    head-major tensors [H,N,D] (inputs resident).  The relayout of one [N,C]
    tensor to or from the head-major layout is timed on its own.  Prints its
    own JSON line; the headline line is the layer's."""
    import numpy as np
    import torch
    from paper_2502_02414_amd import binding as B
    from paper_2502_02414_amd import inputs as I
    from paper_2502_02414_amd.heads import HeadSlicedLayer

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    w = I.WORKLOADS[WORKLOAD]
    N, C, H, M = w.N, w.C, w.H, w.M
    D = C // H
    t0 = time.time()
    bf = torch.bfloat16
    to = lambda a, dt=torch.float32: torch.from_numpy(np.ascontiguousarray(a)).cuda().to(dt)
    x, dY = to(I.make_x(w), bf), to(I.make_grad(w), bf)
    G = to(I.make_head_gumbel(w), bf)
    p = I.make_head_params(w)
    pd = {k: ([float(t) for t in v] if k == "b_t" else to(v, bf if k in ("A", "a") else
                                                          torch.float32)) for k, v in p.items()}
    print(f"[bench] per-head inputs generated in {time.time() - t0:.1f}s", file=sys.stderr,
          flush=True)
    L = HeadSlicedLayer(N, H, D, M, pd, bf, w.tau0, w.tau_min, w.eps, streams=args.head_streams,
                        batched=None if args.head_calls is None else args.head_calls == "batched")
    xh, dYh = L.to_heads(x), L.to_heads(dY)
    del x, dY
    steps, warmup = args.steps, args.warmup
    for _ in range(warmup):
        L.forward(xh, G)
        L.backward(dYh)
    torch.cuda.synchronize()
    # forward / backward split in a pass of its own (events stay out of the
    # timed region)
    ev = [[B.HipEvent() for _ in range(3)] for _ in range(steps)]
    for s in range(steps):
        ev[s][0].record()
        L.forward(xh, G)
        ev[s][1].record()
        L.backward(dYh)
        ev[s][2].record()
    torch.cuda.synchronize()
    fwd = sum(e[0].elapsed_ms(e[1]) for e in ev) / steps
    bwd = sum(e[1].elapsed_ms(e[2]) for e in ev) / steps
    # the timed region; the library brackets the streaming kernel of the
    # slice backward (all heads in one launch) with an event pair per step
    start, end = B.HipEvent(), B.HipEvent()
    kev = [(B.HipEvent(), B.HipEvent()) for _ in range(steps)]
    batched = L.batched
    start.record()
    for s in range(steps):
        if batched:
            B.pa_time_kernel("pa_slice_aggregate_backward", *kev[s])
        L.forward(xh, G)
        L.backward(dYh)
    end.record()
    torch.cuda.synchronize()
    B.pa_time_kernel(None)
    ms = start.elapsed_ms(end) / steps
    kernel_ms = sum(e0.elapsed_ms(e1) for e0, e1 in kev) / steps if batched else None
    if args.copy_calibration:
        src = torch.empty(1 << 28, dtype=torch.float32, device="cuda")  # 1 GiB
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    # one [N,C] tensor to the head-major layout and back
    tmp = torch.empty(N, C, dtype=bf, device="cuda")
    r0, r1 = B.HipEvent(), B.HipEvent()
    r0.record()
    for _ in range(steps):
        B.pa_heads_relayout(xh, tmp, H, to_heads=False)
        B.pa_heads_relayout(tmp, xh, H, to_heads=True)
    r1.record()
    torch.cuda.synchronize()
    relayout_ms = r0.elapsed_ms(r1) / (2 * steps)
    bpp = algo_bytes_per_point(D, M, 2, 2)
    step_bytes = H * N * sum(bpp[n] for n in ("pa_slice_aggregate", "pa_deslice",
                                              "pa_deslice_backward",
                                              "pa_slice_aggregate_backward"))
    gbs = step_bytes / (ms * 1e-3) / 1e9
    out = {
        "metric": "mesh points/sec, per-head sliced Physics-Attention layer fwd+bwd at N=1M, "
                  "C=256 (H=8 heads of D=32), M=32 per head",
        "value": round(N / (ms * 1e-3), 1), "unit": "points/s", "n_gpus": 1, "steps": steps,
        "warmup": warmup, "ms_per_step": round(ms, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": WORKLOAD + "_per_head", "N": N, "C": C, "H": H, "D": D, "M": M,
                   "slicing": "per-head", "layout": "head-major [H,N,D]",
                   "calls": "batched" if L.batched else "per-head", "streams": L.ns,
                   "pass": "forward+backward"},
        "forward_ms": round(fwd, 4), "backward_ms": round(bwd, 4),
        "step_hbm": {"algo_bytes": step_bytes, "achieved_GBs": round(gbs, 1),
                     "frac": round(gbs / HBM_PEAK_GBS, 4)},
        "relayout_ms_per_tensor": round(relayout_ms, 4),
        "relayout_GBs": round(2 * N * C * 2 / (relayout_ms * 1e-3) / 1e9, 1),
    }
    if args.probe:
        # each pass's access pattern alone (pa_stream_probe): the head-major
        # tensors as one head of H N points of D channels, the same bytes in
        # the same 64-byte rows (one grid over all heads' points instead of
        # one per head), each probe after a 1 GiB write
        pdims = B.make_dims(H * N, D, 1, M, w.tau0, w.tau_min, w.eps, B.PA_BF16)
        pout = torch.empty(H * N, D, dtype=bf, device="cuda")
        junk = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
        e0, e1 = B.HipEvent(), B.HipEvent()
        probe = {}
        for c in ("pa_slice_aggregate", "pa_deslice", "pa_deslice_backward",
                  "pa_slice_aggregate_backward"):
            rd = c in ("pa_deslice_backward", "pa_slice_aggregate_backward")
            wr = c in ("pa_deslice", "pa_slice_aggregate_backward")
            pt = []
            for r in range(max(3, steps)):
                junk.fill_(float(r))
                e0.record()
                B.pa_stream_probe(pdims, c, xh, dYh if rd else None, G, pout if wr else None)
                e1.record()
                torch.cuda.synchronize()
                pt.append(e0.elapsed_ms(e1))
            pm = sorted(pt)[len(pt) // 2]
            nb = H * N * bpp[c]
            probe[c] = {"probe_us": round(pm * 1e3, 1),
                        "probe_GBs": round(nb / (pm * 1e-3) / 1e9, 1)}
        out["probe"] = probe
    if kernel_ms:
        kb = H * N * bpp["pa_slice_aggregate_backward"]
        ach = kb / (kernel_ms * 1e-3) / 1e9
        out["roofline"] = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS,
                           "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBS, 4),
                           "traffic": read_traffic("slice_bwd_heads"),
                           "call": "pa_heads_slice_aggregate_backward", "kernel": "slice_bwd (C=32)",
                           "algo_bytes_per_launch": kb, "kernel_ms": round(kernel_ms, 4)}
    print(json.dumps(out), flush=True)


def time_steps(calls, bpp, args, B, torch):
    """Warm-up, a per-call breakdown pass, then the timed region of K whole
    steps of `calls`; in each timed step the library brackets the streaming
    kernel of the dominant call with one event pair (its duration for the
    roofline)."""
    def step(events=None):
        for k, (name, fn) in enumerate(calls):
            if events is not None:
                events[k][0].record()
            fn()
            if events is not None:
                events[k][1].record()

    def event_pair():
        return B.HipEvent(), B.HipEvent()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # Per-call breakdown, in its own pass: an event pair around every call
    # costs the GPU a little idle time at each record, so these events stay
    # out of the timed region.
    per_call = {name: 0.0 for name, _ in calls}
    evs = [[event_pair() for _ in calls] for _ in range(args.steps)]
    for s in range(args.steps):
        step(evs[s])
    torch.cuda.synchronize()
    for s in range(args.steps):
        for k, (name, _) in enumerate(calls):
            per_call[name] += evs[s][k][0].elapsed_ms(evs[s][k][1]) / args.steps
    dom = max((n for n in per_call if bpp[n] > 0), key=lambda n: per_call[n])

    kev = [event_pair() for _ in range(args.steps)]
    start, end = event_pair()
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    start.record()
    for s in range(args.steps):
        B.pa_time_kernel(dom, *kev[s])
        step()
    end.record()
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    B.pa_time_kernel(None)
    return {"dom": dom, "per_call": per_call, "ms_per_step": start.elapsed_ms(end) / args.steps,
            "kernel_ms": sum(e0.elapsed_ms(e1) for e0, e1 in kev) / args.steps,
            "wall_s": t_wall}


def _oracle_rate(oracle, w, x_np, G_np, dY_np, p, target_s):
    """Points/s of the oracle's layer (forward, and backward if the workload
    has one) on the first n points, n sized from a short calibration run so
    that the timed run takes about target_s seconds.  Returns (rate, n, s)."""
    pp = {k: v for k, v in p.items() if v is not None}

    def run(n):
        xs, Gs, dYs = x_np[:n], G_np[:n], dY_np[:n]
        t = time.perf_counter()
        f = oracle.layer_forward(xs, Gs, pp, w.tau0, w.tau_min, w.eps, w.H)
        if w.backward:
            oracle.layer_backward(xs, Gs, pp, w.tau0, w.tau_min, w.eps, w.H, f, dYs)
        return time.perf_counter() - t

    n0 = min(len(x_np), 4096)
    rate0 = n0 / run(n0)
    n = int(min(len(x_np), max(n0, rate0 * target_s)))
    n = (n // 1024) * 1024 or n0
    dt = run(n)
    return n / dt, n, dt


def cpu_baseline(x_np, G_np, dY_np, p, w, target_s: float = 10.0, per_core=None):
    """The oracle, as it stands, on the host cores: the layer in float64 on
    the first n points of the same workload, built on this host with -O3
    -march=native (oracle/build.py's native variant), OpenMP over all the
    cores it may use.  With per_core (a workload), also a one-thread run on
    that workload."""
    import oracle
    oracle.use_variant("native", rebuild=True)
    rate, n, dt = _oracle_rate(oracle, w, x_np, G_np, dY_np, p, target_s)
    passes = "fwd+bwd" if w.backward else "fwd"
    out = {"value": round(rate, 1), "unit": "points/s", "cores": oracle.num_threads(),
           "kind": "oracle",
           "sample": f"first {n} of the {len(x_np)} points of {w.name}, {passes} in float64 "
                     f"({dt:.1f} s; gcc -O3 -march=native, OpenMP)"}
    if per_core is not None:
        from paper_2502_02414_amd import inputs as I
        w3 = per_core
        x3, G3, dY3, p3 = I.make_x(w3), I.make_gumbel(w3), I.make_grad(w3), I.make_params(w3)
        threads = oracle.num_threads()
        oracle.set_num_threads(1)
        try:
            r1, n1, t1 = _oracle_rate(oracle, w3, x3, G3, dY3, p3, target_s / 2)
        finally:
            oracle.set_num_threads(threads)
        out["per_core"] = {"value": round(r1, 1), "unit": "points/s", "cores": 1,
                           "workload": w3.name,
                           "sample": f"first {n1} of the {len(x3)} points of {w3.name}, "
                                     f"fwd+bwd in float64 on one thread ({t1:.1f} s)"}
    return out


if __name__ == "__main__":
    main()

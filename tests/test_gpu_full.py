"""HIP path vs the CPU oracle at the workloads' full sizes, through the C ABI.

* The million-point car-surface workload (N = 1,000,000, C = 256, H = 8,
  M = 32, bf16 storage): the exact inputs and call sequences that bench.py
  times (weights recomputed in every pass, and stored once).  The oracle
  evaluates the whole layer forward + backward in float64 on the host cores
  (about half a minute), so every output tensor is compared in full, by
  relative L2.
* The largest single-layer shape, the aircraft-surface workload (N = 2.5M,
  C = 256, H = 8, M = 64, bf16): the layer must fit and run on one GPU.  The
  oracle computes every quantity that sums over all points (num, den, S, S',
  dS', dS and the token-attention gradients) and the per-point outputs y and
  dx on a seeded sample of rows, which it evaluates one by one from those
  sums; the projection gradients dA, db, da (sums over all points of the
  per-point chain rule) are checked in full at the million-point size only.
"""
import numpy as np
import pytest

import oracle
from paper_2502_02414_amd import inputs as I
from pa_cases import TOL, Gpu, host, make_case, oracle_params, rel_l2, say

pytestmark = pytest.mark.gpu


def check(name, got, ref, dt):
    e = rel_l2(got, ref)
    say(f"  {name:8s} rel_l2 = {e:.3e}  (bar {TOL[dt]:.0e})")
    assert np.isfinite(e) and e <= TOL[dt], (name, e)


def test_full_size_bench_workload():
    w = I.WORKLOADS["car_1m_bf16"]
    say(f"full size {w.name}: N={w.N} C={w.C} H={w.H} M={w.M} {w.dtype}")
    c = make_case(w.N, w.C, w.H, w.M, w.dtype, biases=False, workload=w)
    g = Gpu(c)
    outs = {"recomputed weights": g.layer(), "stored weights": g.layer_w()}
    g.torch.cuda.synchronize()
    say("  gpu layers done; oracle forward + backward ...")
    p = oracle_params(c)
    f = oracle.layer_forward(c.x, c.G, p, c.tau0, c.tau_min, c.eps, c.H)
    gr = oracle.layer_backward(c.x, c.G, p, c.tau0, c.tau_min, c.eps, c.H, f, c.dY)
    for name, out in outs.items():
        say(f" {name}")
        for k in ("num", "den", "S", "Sp", "y"):
            check(k, host(out[k]), f[k], c.dt)
        if "W" in out:
            check("W", host(out["W"]), f["W"], c.dt)
        for k in ("dSp", "dS", "dWq", "dbq", "dWk", "dWv", "dbv", "dx", "dA", "db"):
            check(k, host(out[k]), gr[k], c.dt)
        # the Ada-Temp parameters (a, b_t) as one gradient (as in the per-call tests)
        da = np.concatenate([host(out["da"]).ravel(), host(out["db_t"]).ravel()])
        check("d(a,b_t)", da, np.concatenate([gr["da"].ravel(), [gr["db_t"]]]), c.dt)
        assert float(host(out["dtau0"])[0]) == float(host(out["db_t"])[0])


def test_max_size_layer_fits_and_matches_sampled_rows():
    w = I.WORKLOADS["aircraft_2p5m_bf16"]
    say(f"max size {w.name}: N={w.N} C={w.C} H={w.H} M={w.M} {w.dtype}")
    c = make_case(w.N, w.C, w.H, w.M, w.dtype, workload=w)
    g = Gpu(c)
    out = g.layer()
    g.torch.cuda.synchronize()
    say("  gpu layer done; oracle sums over all points ...")
    p = oracle_params(c)
    W, _, _ = oracle.slice_weights(c.x, c.G, p["A"], p.get("b"), p.get("a"), p.get("b_t", 0.0),
                                   c.tau0, c.tau_min)
    num, den, S = oracle.aggregate(c.x, W, c.eps)
    Sp = oracle.token_attention(S, c.H, p["Wq"], p.get("bq"), p["Wk"], p.get("bk"), p["Wv"],
                                p.get("bv"))
    dSp = oracle.deslice_backward(W, Sp, c.dY)[0]
    att = oracle.token_attention_backward(S, c.H, p["Wq"], p.get("bq"), p["Wk"], p.get("bk"),
                                          p["Wv"], p.get("bv"), None, None, dSp)
    del W
    for k, ref in (("num", num), ("den", den), ("S", S), ("Sp", Sp), ("dSp", dSp),
                   ("dS", att["dS"]), ("dWq", att["dWq"]), ("dWk", att["dWk"]),
                   ("dWv", att["dWv"]), ("dbv", att["dbv"])):
        check(k, host(out[k]), ref, c.dt)
    # per-point outputs on 4096 seeded rows (both ends of the range included)
    rows = np.unique(np.concatenate([
        [0, c.N - 1], np.random.default_rng(2502).integers(0, c.N, 4094)]))
    say(f"  sampled rows: {rows.size}")
    xs, Gs, dYs = c.x[rows], c.G[rows], c.dY[rows]
    Ws, _, _ = oracle.slice_weights(xs, Gs, p["A"], p.get("b"), p.get("a"), p.get("b_t", 0.0),
                                    c.tau0, c.tau_min)
    ys = oracle.deslice(Ws, Sp)
    _, dW_des = oracle.deslice_backward(Ws, Sp, dYs)
    dx_agg, dW_agg = oracle.aggregate_backward(xs, Ws, num, den, att["dS"], c.eps)
    sw = oracle.slice_weights_backward(xs, Gs, p["A"], p.get("b"), p.get("a"), p.get("b_t", 0.0),
                                       c.tau0, c.tau_min, dW_des + dW_agg)
    idx = g.torch.from_numpy(rows).to("cuda")
    check("y[rows]", host(out["y"].index_select(0, idx)), ys, c.dt)
    check("dx[rows]", host(out["dx"].index_select(0, idx)), dx_agg + sw["dx"], c.dt)

"""The oracle's block stack with the GPU path's storage roundings applied
(test helper, not collected by pytest).

The GPU stack (paper_2502_02414_amd/stack.py) stores its point-side
intermediates in the storage dtype (LN1(x), the deslice output, x1,
LN2(x1), GELU of the MLP's pre-activation, every block output, and in the
backward du, dLN2, dx1, dh, dx; with fp32 storage also the pre-activation
and dGELU, which bf16 storage keeps in registers), keeps the token-side tensors in
fp32 (num, den, S, S_proj, S', dS', dS_proj, dS) and folds Algorithm 1's
Project step into the slice parameters (A' = Wp A and a' = Wp a, in the
storage dtype).  ``stack_model`` evaluates the oracle's own steps (its
LayerNorm, GELU, slice weights, aggregation, token attention, deslice and
their chain rules, in float64) in that folded form, rounding exactly those
tensors to their storage type.  With no rounding it equals
oracle.stack_forward / stack_backward (the Project folding is exact when
every den_j >= eps); with rounding, its distance to them is what the
storage types alone cost: the parity bars of the stack tests are derived
from it.
"""
from __future__ import annotations

import numpy as np

import oracle
from paper_2502_02414_amd import inputs as I

ATTN = ("Wq", "bq", "Wk", "bk", "Wv", "bv", "Wo", "bo")
GRADS = ("dW2", "db2", "dW1", "db1", "dln2_g", "dln2_b", "dWq", "dbq", "dWk", "dWv", "dbv",
         "dWo", "dbo", "dWp", "dbp", "dA", "db", "dln1_g", "dln1_b")


def _rounders(dt, rnd, jitter=0.0, seed=0):
    """(storage rounding, fp32 rounding); with jitter, every value is first
    moved by a relative N(0, jitter^2) step (a stand-in for the last-bit
    differences of another evaluation order)."""
    f64 = lambda a: np.asarray(a, dtype=np.float64)
    if not rnd:
        return f64, f64
    rng = np.random.default_rng(seed)
    jit = (lambda a: f64(a) * (1.0 + jitter * rng.standard_normal(np.shape(a)))) if jitter \
        else f64
    f32 = lambda a: np.asarray(jit(a), dtype=np.float32).astype(np.float64)
    if dt == "bf16":
        return (lambda a: I.round_bf16(np.asarray(jit(a), dtype=np.float32)).astype(np.float64),
                f32)
    return f32, f32


def stack_model(x, dY, Gs, ps, tau0, tau_min, eps, H, dt, rnd=True, jitter=0.0, seed=0):
    """Forward + backward of the stack.  Returns (out, dx, [grads per layer])
    with the gradients named as in oracle.stack_backward."""
    R, F = _rounders(dt, rnd, jitter, seed)  # storage-dtype and fp32 rounding
    # bf16: the MLP's first product and its activation are one kernel
    # (pa_mlp_up): u and dY W2^T stay in fp32 registers, only GELU(u) and
    # dU are stored; fp32 storage stores u and dY W2^T (pa_gemm, pa_gelu)
    fused = dt == "bf16"
    x = np.asarray(x, dtype=np.float64)
    caches = []
    for G, p in zip(Gs, ps):
        Wp, bp, A, a = (np.asarray(p[k], dtype=np.float64) for k in ("Wp", "bp", "A", "a"))
        h = R(oracle.layernorm(x, p["ln1_g"], p["ln1_b"])[0])
        Af, af = R(Wp @ A), R(Wp @ a)
        bf = F(np.asarray(p["b"], dtype=np.float64) + bp @ A)
        bt = float(p.get("b_t", 0.0)) + float(F(bp @ a))
        W, _, _ = oracle.slice_weights(h, G, Af, bf, af, bt, tau0, tau_min)
        num, den, S = map(F, oracle.aggregate(h, W, eps))
        S_proj = F(S @ Wp + bp)
        att = [p.get(k) for k in ATTN]
        Sp = F(oracle.token_attention(S_proj, H, *att))
        x1 = R(x + R(oracle.deslice(W, Sp)))
        h2 = R(oracle.layernorm(x1, p["ln2_g"], p["ln2_b"])[0])
        u = h2 @ np.asarray(p["W1"], dtype=np.float64) + p["b1"]
        if not fused:
            u = R(u)
        gu = R(oracle.gelu(u))
        x2 = R(x1 + gu @ np.asarray(p["W2"], dtype=np.float64) + p["b2"])
        caches.append(dict(x=x, h=h, Af=Af, bf=bf, af=af, bt=bt, W=W, num=num, den=den, S=S,
                           S_proj=S_proj, Sp=Sp, x1=x1, h2=h2, u=u, gu=gu))
        x = x2
    out = x
    dy = R(dY)
    grads = [None] * len(ps)
    for l in reversed(range(len(ps))):
        p, c = ps[l], caches[l]
        Wp, bp, A, a = (np.asarray(p[k], dtype=np.float64) for k in ("Wp", "bp", "A", "a"))
        W1, W2 = (np.asarray(p[k], dtype=np.float64) for k in ("W1", "W2"))
        g = {"dW2": c["gu"].T @ dy, "db2": dy.sum(axis=0)}
        dgu = dy @ W2.T
        du = R(oracle.gelu_backward(c["u"], dgu if fused else R(dgu)))
        g["dW1"], g["db1"] = c["h2"].T @ du, du.sum(axis=0)
        dh2 = R(du @ W1.T)
        dx1_ln, g["dln2_g"], g["dln2_b"] = oracle.layernorm_backward(c["x1"], p["ln2_g"], dh2)
        dx1 = R(dx1_ln + dy)
        dSp, dW_des = oracle.deslice_backward(c["W"], c["Sp"], dx1)
        att = oracle.token_attention_backward(c["S_proj"], H, *[p.get(k) for k in ATTN], F(dSp))
        g.update({k: v for k, v in att.items() if k != "dS"})
        dS_proj = F(att["dS"])
        dS = F(dS_proj @ Wp.T)
        dx_agg, dW_agg = oracle.aggregate_backward(c["h"], c["W"], c["num"], c["den"], dS, eps)
        sw = oracle.slice_weights_backward(c["h"], Gs[l], c["Af"], c["bf"], c["af"], c["bt"],
                                           tau0, tau_min, dW_des + dW_agg)
        dh = R(dx_agg + sw["dx"])
        dAf, dbf, daf, dbtf = F(sw["dA"]), F(sw["db"]), F(sw["da"]), float(F(sw["db_t"]))
        # the folding's chain rule (Project: x_proj = h Wp + bp)
        g["dWp"] = dAf @ A.T + np.outer(daf, a) + c["S"].T @ dS_proj
        g["dbp"] = A @ dbf + dbtf * a + dS_proj.sum(axis=0)
        g["dA"] = Wp.T @ dAf + np.outer(bp, dbf)
        g["da"] = Wp.T @ daf + bp * dbtf
        g["db"], g["db_t"] = dbf, dbtf
        dx_ln, g["dln1_g"], g["dln1_b"] = oracle.layernorm_backward(c["x"], p["ln1_g"], dh)
        grads[l] = g
        dy = R(dx_ln + dx1)
    return out, dy, grads


def _distance(a, b):
    """Per-output relative L2 distance of stack results b from a, keyed
    "out", "dx", (layer, grad name) and (layer, "d(a,b_t)")."""
    from pa_cases import rel_l2
    (out_a, dx_a, g_a), (out_b, dx_b, g_b) = a, b
    e = {"out": rel_l2(out_b, out_a), "dx": rel_l2(dx_b, dx_a)}
    for l, (g, r) in enumerate(zip(g_b, g_a)):
        for k in GRADS:
            if k in r:
                e[(l, k)] = rel_l2(g[k], r[k])
        e[(l, "d(a,b_t)")] = rel_l2(np.concatenate([np.ravel(g["da"]), [g["db_t"]]]),
                                    np.concatenate([np.ravel(r["da"]), [r["db_t"]]]))
    return e


def envelope(x, dY, Gs, ps, tau0, tau_min, eps, H, dt, ref_out, ref_dx, ref_grads):
    """Relative L2 distance of the rounded model from the exact oracle stack,
    per output."""
    model = stack_model(x, dY, Gs, ps, tau0, tau_min, eps, H, dt)
    return _distance((ref_out, ref_dx, ref_grads), model)


# Relative size of the differences between two evaluation orders before a
# value is rounded to bf16 (an fp32 evaluation of a LayerNorm row or of a
# K <= 1024 product differs from float64 by about this much; bf16's own
# rounding step is 2^-8).
JITTER = 5e-7


def flip_spread(x, dY, Gs, ps, tau0, tau_min, eps, H, dt, log=None):
    """Relative L2 distance between two rounded evaluations whose values
    differ by a relative JITTER before every rounding, per output: how much
    the storage roundings' flips alone move each output.  Where it exceeds
    the parity bar, no evaluation with that storage type pins the output."""
    a = stack_model(x, dY, Gs, ps, tau0, tau_min, eps, H, dt, jitter=JITTER, seed=1)
    if log:
        log("  first jittered evaluation done")
    b = stack_model(x, dY, Gs, ps, tau0, tau_min, eps, H, dt, jitter=JITTER, seed=2)
    return _distance(a, b)

"""Block-stack primitives and the stack runner vs the CPU oracle, through the
C ABI.

Each primitive is compared with the oracle's function on the same stored
values (LayerNorm with the fused residual add, its backward, GELU), or with
its plain definition in float64 numpy (the GEMM, the column sums, the
Project folding algebra), at relative L2 1e-5 in fp32 and 2e-2 in bf16.

The stack runner (LN -> Physics-Attention with the folded Project step ->
MLP, residual adds, several blocks) is compared with oracle.stack_forward /
stack_backward, which applies the Project step explicitly.  The stack
stores its point-side intermediates in the storage dtype, and those
roundings alone move the exact result.  tests/stack_rounding.py evaluates
the oracle's own stack with exactly those roundings: its distance from the
exact stack (the envelope) and the distance between two such evaluations
whose values differ in the last bits before each rounding (the flip spread)
are measured per output tensor on the CPU, on the same inputs.  An output
is held to max(plain bar, 2 x envelope) (plain bars: 1e-5 fp32, 2e-2
bf16); with bf16 storage only when its flip spread is below 2e-2, for
otherwise no evaluation with bf16 storage can pin it, and it is checked for
finiteness.  That happens in bf16 where a block's Ada-Temp leaves points at
the temperature floor tau_min: the softmax is 1/tau_min = 100 times
sharper, the slice-parameter gradients (dA, db, da, b_t) move by tens of
percent when only the block's input LN1(x) or the folded A' is rounded to
bf16, and in a deep stack the backward carries that into every gradient
below the block.  Without clamped points (the Ada-Temp projection scaled by
0.05) and in fp32 every output is pinned.
"""
import numpy as np
import pytest

import oracle
from paper_2502_02414_amd import binding as B
from paper_2502_02414_amd import inputs as I
from pa_cases import TOL, dev, host, rel_l2, say

pytestmark = pytest.mark.gpu



def check(name, got, ref, bar):
    e = rel_l2(got, ref)
    say(f"  {name:10s} rel_l2 = {e:.3e}  (bar {bar:.0e})")
    assert np.isfinite(e) and e <= bar, (name, e, bar)


def _rnd(dt, *shape, scale=1.0, seed=0, shift=0.0):
    """Seeded values representable in the storage dtype (rounded last)."""
    a = (scale * np.random.default_rng(seed).standard_normal(shape) + shift).astype(np.float32)
    return I.round_bf16(a) if dt == "bf16" else a


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("C", [64, 256])
@pytest.mark.parametrize("residual", [False, True])
def test_layernorm(dt, C, residual):
    say(f"layernorm {dt} C={C} residual={residual}")
    import torch
    N = 1037
    x, r = _rnd(dt, N, C, scale=2.0, seed=1, shift=0.5), _rnd(dt, N, C, seed=2)
    g, b = 1 + 0.1 * _rnd("f32", C, seed=3), 0.1 * _rnd("f32", C, seed=4)
    xd, rd = dev(x, dt), dev(r, dt)
    y, mean, rstd = dev(np.zeros((N, C), np.float32), dt), torch.empty(N, device="cuda"), \
        torch.empty(N, device="cuda")
    xs = dev(np.zeros((N, C), np.float32), dt) if residual else None
    B.pa_layernorm(xd, y, mean, rstd, g=dev(g), b=dev(b), r=rd if residual else None, xs=xs)
    s = x.astype(np.float64)
    if residual:
        s = (x + r).astype(np.float32)
        s = I.round_bf16(s) if dt == "bf16" else s
        np.testing.assert_array_equal(host(xs), s)   # the rounded sum, exactly
    ref, m_ref, r_ref = oracle.layernorm(s, g, b)
    check("y", host(y), ref, TOL[dt])
    check("mean", host(mean), m_ref, 1e-5)
    check("rstd", host(rstd), r_ref, 1e-5)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("C", [64, 256])
def test_layernorm_backward(dt, C):
    say(f"layernorm_backward {dt} C={C}")
    import torch
    N = 2111
    x = _rnd(dt, N, C, scale=2.0, seed=5)
    dy, dres = _rnd(dt, N, C, seed=6), _rnd(dt, N, C, seed=7)
    g, b = 1 + 0.1 * _rnd("f32", C, seed=8), 0.1 * _rnd("f32", C, seed=9)
    xd = dev(x, dt)
    y, mean, rstd = dev(np.zeros((N, C), np.float32), dt), torch.empty(N, device="cuda"), \
        torch.empty(N, device="cuda")
    B.pa_layernorm(xd, y, mean, rstd, g=dev(g), b=dev(b))
    dx = dev(np.zeros((N, C), np.float32), dt)
    dg, db = torch.empty(C, device="cuda"), torch.empty(C, device="cuda")
    ws = torch.empty(1024 * 2 * C, device="cuda")
    B.pa_layernorm_backward(xd, mean, rstd, dev(dy, dt), dx, g=dev(g), dres=dev(dres, dt), dg=dg,
                            db=db, ws=ws)
    rdx, rdg, rdb = oracle.layernorm_backward(x, g, dy)
    check("dx", host(dx), rdx + dres, TOL[dt])
    check("dg", host(dg), rdg, TOL[dt])
    check("db", host(db), rdb, TOL[dt])


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_gelu(dt):
    say(f"gelu {dt}")
    n = 4096 * 12
    x = _rnd(dt, n, scale=3.0, seed=10)
    dy = _rnd(dt, n, seed=11)
    xd = dev(x, dt)
    y, dx = dev(np.zeros(n, np.float32), dt), dev(np.zeros(n, np.float32), dt)
    B.pa_gelu(xd, y)
    B.pa_gelu_backward(xd, dev(dy, dt), dx)
    check("gelu", host(y), oracle.gelu(x), TOL[dt])
    check("dgelu", host(dx), oracle.gelu_backward(x, dy), TOL[dt])


MLP_UP = [  # N, K, F: ragged last block (128 points per block), every K served
    (1000, 64, 256), (77, 128, 512), (4099, 256, 1024), (1, 256, 1024)]


@pytest.mark.parametrize("case", MLP_UP, ids=[f"N{c[0]}-K{c[1]}-F{c[2]}" for c in MLP_UP])
def test_mlp_up(case):
    """The MLP's first product with GELU in one kernel, and its chain rule
    with the pre-activation recomputed, against the oracle's GELU and its
    derivative applied to the float64 products of the same bf16 values."""
    import torch
    N, K, F = case
    say(f"mlp_up N={N} K={K} F={F}")
    X, dY = _rnd("bf16", N, K, seed=20), _rnd("bf16", N, K, seed=21)
    W1 = _rnd("bf16", K, F, scale=K ** -0.5, seed=22)
    W2 = _rnd("bf16", F, K, scale=F ** -0.5, seed=23)
    b1 = _rnd("f32", F, scale=0.1, seed=24)
    ws = torch.empty(2 * F * K, dtype=torch.uint8, device="cuda")
    Xd, W1d, b1d = dev(X, "bf16"), dev(W1, "bf16"), dev(b1)
    G = dev(np.zeros((N, F), np.float32), "bf16")
    dU = dev(np.zeros((N, F), np.float32), "bf16")
    B.pa_mlp_up(Xd, W1d, b1d, G, ws)
    B.pa_mlp_up_backward(Xd, W1d, b1d, dev(dY, "bf16"), dev(W2, "bf16"), dU, ws)
    u = X.astype(np.float64) @ W1.astype(np.float64) + b1
    dg = dY.astype(np.float64) @ W2.astype(np.float64).T
    ref_g, ref_du = oracle.gelu(u), oracle.gelu_backward(u, dg)
    check("G", host(G), ref_g, TOL["bf16"])
    check("dU", host(dU), ref_du, TOL["bf16"])
    # the kernels round a fp32 accumulation once: within a few bf16 steps of
    # the exact values, element by element
    for name, got, ref in (("G", host(G), ref_g), ("dU", host(dU), ref_du)):
        err = np.abs(got - ref) / (np.abs(ref) + 1e-3 * np.abs(ref).max())
        say(f"  {name:10s} max element error {err.max():.2e} (bf16 step 3.9e-3)")
        assert err.max() < 2e-2, (name, err.max())


GEMMS = [  # m, n, k, transA, transB, in dtype, out dtype, bias, residual
    (1000, 96, 64, False, False, "f32", "f32", True, False),
    (1000, 96, 64, False, True, "f32", "f32", False, True),
    (64, 96, 1000, True, False, "f32", "f32", False, False),
    (1003, 256, 64, False, False, "bf16", "bf16", True, True),
    (256, 64, 3001, True, False, "bf16", "f32", False, False),
    (3001, 64, 256, False, True, "bf16", "bf16", False, False),
    # a weight-gradient shape long enough for the split over K (18 chunks + a rest)
    (256, 64, 300001, True, False, "bf16", "f32", False, False),
]


@pytest.mark.parametrize("case", GEMMS, ids=[f"{c[0]}x{c[1]}x{c[2]}-{c[3]:d}{c[4]:d}-{c[5]}-{c[6]}"
                                             for c in GEMMS])
def test_gemm(case):
    m, n, k, tA, tB, ti, to, bias, resid = case
    say(f"gemm {case}")
    A = _rnd(ti, *((k, m) if tA else (m, k)), seed=12)
    Bm = _rnd(ti, *((n, k) if tB else (k, n)), seed=13)
    bv = _rnd("f32", n, seed=14) if bias else None
    Cr = _rnd(to, m, n, seed=15) if resid else None
    ws = dev(np.zeros(16 << 18, np.float32))
    ref = (A.T if tA else A).astype(np.float64) @ (Bm.T if tB else Bm).astype(np.float64)
    if bias:
        ref = ref + bv
    if resid:
        ref = ref + Cr
    # untuned (the heuristic's first algorithm), then tuned by
    # pa_gemm_prepare, then the tuned algorithm through pa_gemm
    for prepare in (False, True, False):
        D = dev(np.zeros((m, n), np.float32), to)
        B.pa_gemm(dev(A, ti), dev(Bm, ti), D, transA=tA, transB=tB,
                  bias=dev(bv) if bias else None, beta=1.0 if resid else 0.0,
                  C=dev(Cr, to) if resid else None, ws=ws, prepare=prepare)
        check(f"D{' (prepare)' if prepare else ''}", host(D), ref,
              TOL[to] if to == "bf16" else 1e-5)


def test_colsum():
    import torch
    for dt, (N, C) in (("f32", (5003, 96)), ("bf16", (3001, 1024))):
        x = _rnd(dt, N, C, seed=16)
        out = torch.empty(C, device="cuda")
        ws = torch.empty(1024 * C, device="cuda")
        B.pa_colsum(dev(x, dt), out, ws)
        check(f"colsum {dt}", host(out), x.astype(np.float64).sum(axis=0), 1e-5)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_project_fold_states_and_backward(dt):
    """The folding algebra against its definition (float64 numpy)."""
    say(f"project {dt}")
    import torch
    C, M, H = 64, 16, 4
    rng = np.random.default_rng(17)
    r = lambda *s: (0.3 * rng.standard_normal(s)).astype(np.float32)
    Wp, bp, A, b, a = r(C, C), r(C), r(C, M), r(M), r(C)
    S, dSp = r(M, C), r(M, C)
    dAf, dbf, daf, dbtf = r(C, M), r(M), r(C), r(1)
    dims = B.make_dims(100, C, H, M, 0.5, 0.01, 1e-5, B.PA_BF16 if dt == "bf16" else B.PA_F32)
    Af, af = dev(np.zeros((C, M), np.float32), dt), dev(np.zeros(C, np.float32), dt)
    bf, btf = torch.empty(M, device="cuda"), torch.empty(1, device="cuda")
    B.pa_project_fold(dims, dev(Wp), dev(bp), dev(A), dev(b), dev(a), Af, bf, af, btf)
    W64, bp64, A64, a64 = (v.astype(np.float64) for v in (Wp, bp, A, a))
    bar = TOL[dt] if dt == "bf16" else 1e-5
    check("A'", host(Af), W64 @ A64, bar)
    check("a'", host(af), W64 @ a64, bar)
    check("b'", host(bf), b + bp64 @ A64, 1e-5)
    check("b_t'", host(btf), [bp64 @ a64], 1e-5)
    Sproj = torch.empty(M, C, device="cuda")
    B.pa_project_states(dims, dev(S), dev(Wp), dev(bp), Sproj)
    check("S_proj", host(Sproj), S.astype(np.float64) @ W64 + bp64, 1e-5)
    f32 = lambda *s: torch.empty(*s, device="cuda")
    dWp, dbp, dS, dA, db_, da, dbt = f32(C, C), f32(C), f32(M, C), f32(C, M), f32(M), f32(C), f32(1)
    keep = {k: dev(v) for k, v in (("dA", dAf), ("db", dbf), ("da", daf), ("db_t", dbtf))}
    folded = B.make_slice_grads(**keep)  # raw pointers: the tensors must outlive the call
    B.pa_project_backward(dims, dev(Wp), dev(bp), dev(A), dev(a), dev(S), dev(dSp), folded, dWp,
                          dbp, dS, B.make_slice_grads(dA=dA, db=db_, da=da, db_t=dbt))
    S64, dSp64 = S.astype(np.float64), dSp.astype(np.float64)
    check("dWp", host(dWp), dAf @ A64.T + np.outer(daf, a64) + S64.T @ dSp64, 1e-5)
    check("dbp", host(dbp), A64 @ dbf + dbtf[0] * a64 + dSp64.sum(axis=0), 1e-5)
    check("dA", host(dA), W64.T @ dAf + np.outer(bp64, dbf), 1e-5)
    check("da", host(da), W64.T @ daf + bp64 * dbtf[0], 1e-5)
    check("dS", host(dS), dSp64 @ W64.T, 1e-5)
    np.testing.assert_array_equal(host(db_), dbf)
    np.testing.assert_array_equal(host(dbt), dbtf)


# ---------------------------------------------------------------------------
# The stack runner
# ---------------------------------------------------------------------------

def stack_case(N, C, H, M, L, dt, geometry="normal", a_scale=1.0):
    w = I.small("stack", N, C, H, M, dt, geometry=geometry)
    x, dY = I.make_x(w, N), I.make_grad(w, N)
    ps = [I.make_block_params(w, l) for l in range(L)]
    for p in ps:  # the Ada-Temp projection, scaled (values kept in the storage dtype)
        a = (p["a"] * np.float32(a_scale)).astype(np.float32)
        p["a"] = I.round_bf16(a) if dt == "bf16" else a
    Gs = [I.make_layer_gumbel(w, l, N) for l in range(L)]
    return w, x, dY, ps, Gs


def device_params(ps, dt):
    out = []
    for p in ps:
        q = {}
        for k, v in p.items():
            if k == "b_t":
                q[k] = float(v)
            else:
                q[k] = dev(v, dt if k in ("W1", "W2") else "f32")
        out.append(q)
    return out


STACKS = [
    # N, C, H, M, blocks, dtype, Ada-Temp scale
    (2000, 64, 4, 16, 2, "f32", 1.0),
    (2000, 64, 4, 16, 2, "bf16", 0.05),
    (3001, 256, 8, 32, 2, "bf16", 0.05),
    # the generator's Ada-Temp: about a third of the points at tau_min
    (2000, 64, 4, 16, 2, "bf16", 1.0),
    (3001, 256, 8, 32, 2, "bf16", 1.0),
]


def _compare_stack(N, C, H, M, L, dt, a_scale, geometry="normal"):
    from paper_2502_02414_amd.stack import BlockStack
    import stack_rounding as SR
    import torch
    w, x, dY, ps, Gs = stack_case(N, C, H, M, L, dt, geometry=geometry, a_scale=a_scale)
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    st = BlockStack(N, C, H, M, device_params(ps, dt), tdt, w.tau0, w.tau_min, w.eps)
    out = st.forward(dev(x, dt), [dev(G, dt) for G in Gs])
    dx, grads = st.backward(dev(dY, dt))
    torch.cuda.synchronize()
    say("  GPU stack done; oracle stack and its rounded evaluation on the CPU")
    ref, caches = oracle.stack_forward(x, Gs, ps, w.tau0, w.tau_min, w.eps, H)
    for c in caches:  # the folded states are exact for den >= eps
        assert np.all(c["pa"]["den"] >= w.eps)
    clamped = [float(np.mean(c["pa"]["t"] <= w.tau_min)) for c in caches]
    say(f"  points at tau_min per block: {np.round(clamped, 2).tolist()}")
    rdx, rgr = oracle.stack_backward(dY, Gs, ps, w.tau0, w.tau_min, w.eps, H, caches)
    say("  oracle stack done")
    env = SR.envelope(x, dY, Gs, ps, w.tau0, w.tau_min, w.eps, H, dt, ref, rdx, rgr)
    say("  rounded evaluation done")
    # (fp32 storage: the roundings are at the level of the evaluation's own
    # last bits, and every output is pinned)
    spread = SR.flip_spread(x, dY, Gs, ps, w.tau0, w.tau_min, w.eps, H, dt, log=say) \
        if dt == "bf16" else None
    unpinned = []

    def cmp(key, name, got, want):
        if spread is not None and spread[key] > TOL[dt]:
            say(f"  {name:10s} not pinned (flip spread {spread[key]:.2e}, envelope "
                f"{env[key]:.2e}); finite")
            assert np.all(np.isfinite(got)), name
            unpinned.append((key, name))
            return
        check(name, got, want, max(TOL[dt], 2.0 * env[key]))

    cmp("out", "out", host(out), ref)
    cmp("dx", "dx", host(dx), rdx)
    for l in range(L):
        say(f" layer {l}")
        for k in SR.GRADS:
            cmp((l, k), k, host(grads[l][k]), rgr[l][k])
        ga = np.concatenate([host(grads[l]["da"]).ravel(), host(grads[l]["db_t"]).ravel()])
        cmp((l, "d(a,b_t)"), "d(a,b_t)", ga,
            np.concatenate([rgr[l]["da"].ravel(), [rgr[l]["db_t"]]]))
        # the key bias shifts a whole score row: its gradient is 0 up to rounding
        assert np.linalg.norm(host(grads[l]["dbk"])) <= \
            TOL[dt] * np.linalg.norm(host(grads[l]["dbq"]))
    say(f"  {len(unpinned)} outputs not pinned")
    # the forward output and the input gradient are always pinned
    assert "out" not in [k for k, _ in unpinned] and "dx" not in [k for k, _ in unpinned]
    if a_scale < 1.0 or dt == "f32":
        assert not unpinned
    return clamped


@pytest.mark.parametrize("shape", STACKS, ids=[f"N{s[0]}-C{s[1]}-M{s[3]}-L{s[4]}-{s[5]}-a{s[6]}"
                                               for s in STACKS])
def test_block_stack(shape):
    """GPU stack (folded Project) vs the oracle stack (explicit Project)."""
    say(f"stack {shape}")
    clamped = _compare_stack(*shape)
    if shape[6] < 1.0:
        assert max(clamped) == 0.0
    else:
        assert max(clamped) > 0.2


def test_block_stack_eight_blocks():
    """The configuration of the full-size stack (8 blocks, C = 256, H = 8,
    M = 64, bf16, the aircraft-surface inputs and the generator's weights)
    at N = 50,000 points (several 16-point tiles per wave in every streaming
    pass), every output and gradient against the oracle."""
    say("stack 8 blocks, N=50000 C=256 H=8 M=64 bf16 (aircraft surface)")
    _compare_stack(50000, 256, 8, 64, 8, "bf16", 1.0, geometry="aircraft")


def test_block_stack_full_size():
    """The 8-block stack at N = 2.5M points (C = 256, H = 8, M = 64, bf16),
    forward and backward on one GPU.  No oracle runs 8 such layers at this
    size; checked: it fits and runs, every output and gradient is finite,
    the first LayerNorm (row-local) matches the oracle on sampled rows, and
    the gradients are nonzero."""
    from paper_2502_02414_amd.stack import BlockStack
    import torch
    w = I.WORKLOADS["aircraft_2p5m_bf16"]
    N, C, H, M, L = w.N, w.C, w.H, w.M, 8
    say(f"stack full size: N={N} C={C} H={H} M={M} L={L} bf16")
    x = I.make_x(w)
    xd = dev(x, "bf16")
    ps = [I.make_block_params(w, l) for l in range(L)]
    Gs = [dev(I.make_layer_gumbel(w, l), "bf16") for l in range(L)]
    say("  inputs on the GPU")
    st = BlockStack(N, C, H, M, device_params(ps, "bf16"), torch.bfloat16, w.tau0, w.tau_min,
                    w.eps)
    e0, e1, e2 = (B.HipEvent() for _ in range(3))
    e0.record()
    out = st.forward(xd, Gs)
    e1.record()
    dx, grads = st.backward(dev(I.make_grad(w), "bf16"))
    e2.record()
    torch.cuda.synchronize()
    say(f"  forward {e0.elapsed_ms(e1):.1f} ms, backward {e1.elapsed_ms(e2):.1f} ms "
        f"(first call: includes hipBLASLt's algorithm choice); "
        f"{torch.cuda.max_memory_allocated() / 2**30:.1f} GiB peak")
    assert torch.isfinite(out).all() and torch.isfinite(dx).all()
    for l in range(L):
        for k, v in grads[l].items():
            assert torch.isfinite(v).all(), (l, k)
        assert float(grads[l]["dW1"].abs().max()) > 0 and float(grads[l]["dA"].abs().max()) > 0
    rows = np.unique(np.concatenate([[0, N - 1], np.random.default_rng(5).integers(0, N, 2046)]))
    idx = torch.from_numpy(rows).cuda()
    ref, _, _ = oracle.layernorm(x[rows], ps[0]["ln1_g"], ps[0]["ln1_b"])
    check("LN1 rows", host(st.caches[0]["h"].index_select(0, idx)), ref, TOL["bf16"])


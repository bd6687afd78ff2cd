"""HIP path vs the CPU oracle, element by element, through the C ABI.

Each entry point of include/pa.h is fed the same seeded inputs as the oracle
and compared by relative L2 per output tensor: <= 1e-5 for fp32 storage and
<= 2e-2 for bf16 storage with fp32 accumulation.  Shapes span several
16-point tiles with a ragged tail, ragged slice blocks (M not a multiple of
16), M = 1, missing noise / Ada-Temp, the denominator floor, the layer
configurations of the benchmark suite, and sizes with several tiles per
wave (the streaming passes' multi-tile pipeline).
"""
import numpy as np
import pytest

import oracle
from pa_cases import TOL, Gpu, dev, host, make_case, oracle_layer, oracle_params, rel_l2, say

pytestmark = pytest.mark.gpu

SHAPES = [
    # N, C, H, M, dtype
    (1000, 32, 2, 5, "f32"),
    (4096, 64, 4, 16, "f32"),
    (2049, 128, 8, 64, "f32"),
    (3001, 256, 8, 32, "bf16"),
    (777, 64, 4, 33, "bf16"),
    (257, 128, 8, 1, "f32"),
    (517, 256, 8, 64, "bf16"),
    # several 16-point tiles per wave: the streaming passes' register
    # pipeline (a tile's stage reloaded while the previous tile computes)
    (66013, 256, 8, 32, "bf16"),
    (50003, 256, 8, 64, "bf16"),
    (40007, 128, 8, 32, "f32"),
    # the 128 x 128 grid workload's shape (fp32, M = 64: two waves per CU in
    # the backward, several tiles each)
    (16384, 128, 8, 64, "f32"),
    # the block-cooperative slice backward (bf16, C = 256, 33..64 slices):
    # three slice blocks over several tiles; one block with a ragged tile
    (20011, 256, 8, 48, "bf16"),
    (33, 256, 8, 50, "bf16"),
    # channel counts between the kernels' widths (rows of C channels on the
    # kernels of the next width up, zero table columns): C = 16, 48, 80, 96,
    # 160, 208, odd head widths, token projections with a 16-column tail
    (777, 16, 2, 7, "f32"),
    (1000, 48, 4, 20, "bf16"),
    (1203, 80, 5, 12, "f32"),
    (2049, 96, 8, 64, "f32"),
    (3001, 160, 8, 40, "bf16"),
    (5003, 208, 8, 33, "bf16"),
    # narrow rows (bf16 rows of 64 bytes or less: the pass bound by
    # instruction issue, with the biases and dden as the contractions'
    # starting values) with padded slices (M not a multiple of 16)
    (3001, 32, 2, 20, "bf16"),
    (777, 16, 1, 7, "bf16"),
]
IDS = [f"N{n}-C{c}-H{h}-M{m}-{d}" for n, c, h, m, d in SHAPES]


def check(name, gpu, ref, dt, tol=None):
    e = rel_l2(host(gpu) if not isinstance(gpu, np.ndarray) else gpu, ref)
    bar = TOL[dt] if tol is None else tol
    say(f"  {name:8s} rel_l2 = {e:.3e}  (bar {bar:.0e})")
    assert np.isfinite(e) and e <= bar, (name, e, bar)


def check_ada_temp(out, ref, dt, tol=None):
    """The Ada-Temp Linear (Eq. 3) has parameters (a, b_t); its gradient is
    checked as one tensor [da, db_t].  db_t alone is a sum over points of dt_i
    of both signs whose value is a fraction of a percent of sum |dt_i|, so on
    its own its relative error is the per-point error times that condition
    number."""
    g = np.concatenate([host(out["da"]).ravel(), host(out["db_t"]).ravel()])
    r = np.concatenate([np.asarray(ref["da"]).ravel(), [ref["db_t"]]])
    check("d(a,b_t)", g, r, dt, tol)


def check_key_bias(gpu_dbk, gpu_dbq, dt="f32"):
    """The key bias shifts every score of a row by the same q.b_k, which the
    row softmax cancels (Eq. 2): dbk is exactly 0.  Relative error against a
    zero reference is meaningless, so bound |dbk| by the scale of dbq."""
    a, scale = np.linalg.norm(host(gpu_dbk)), np.linalg.norm(host(gpu_dbq))
    say(f"  dbk      |dbk|/|dbq| = {a / max(scale, 1e-30):.3e}")
    assert a <= TOL[dt] * max(scale, 1e-30)


@pytest.fixture(scope="module")
def cases():
    return {}


def get_case(cases, shape, **kw):
    key = (shape, tuple(sorted(kw.items())))
    if key not in cases:
        N, C, H, M, dt = shape
        c = make_case(N, C, H, M, dt, **kw)
        cases[key] = (c, Gpu(c), oracle_layer(c))
    return cases[key]


@pytest.mark.parametrize("shape", SHAPES, ids=IDS)
def test_slice_weights(cases, shape):
    say(f"slice_weights {shape}")
    c, g, (f, _) = get_case(cases, shape)
    W, tau = g.slice_weights()
    check("W", W, f["W"], c.dt)
    check("tau", tau, f["tau"], c.dt)
    Wh = host(W)
    assert np.abs(Wh.sum(1) - 1).max() < 1e-5


@pytest.mark.parametrize("shape", SHAPES, ids=IDS)
def test_slice_aggregate(cases, shape):
    say(f"slice_aggregate {shape}")
    c, g, (f, _) = get_case(cases, shape)
    num, den, S = g.aggregate()
    check("num", num, f["num"], c.dt)
    check("den", den, f["den"], c.dt)
    check("S", S, f["S"], c.dt)


@pytest.mark.parametrize("shape", SHAPES, ids=IDS)
def test_token_attention(cases, shape):
    say(f"token_attention {shape}")
    c, g, (f, _) = get_case(cases, shape)
    S = g.torch.from_numpy(f["S"].astype(np.float32)).cuda()
    Sp = g.attention(S)
    p = oracle_params(c)
    ref = oracle.token_attention(S.cpu().numpy(), c.H, p["Wq"], p.get("bq"), p["Wk"],
                                 p.get("bk"), p["Wv"], p.get("bv"), p.get("Wo"), p.get("bo"))
    check("Sp", Sp, ref, "f32")


def test_token_attention_output_projection(cases):
    shape = (600, 64, 4, 16, "f32")
    c, g, (f, _) = get_case(cases, shape, out_proj=True)
    S = g.torch.from_numpy(f["S"].astype(np.float32)).cuda()
    Sp = g.attention(S)
    check("Sp", Sp, f["Sp"], "f32")
    dSp = g.torch.from_numpy(np.asarray(f["S"][::-1], dtype=np.float32).copy()).cuda()
    ga = g.attention_backward(S, dSp)
    p = oracle_params(c)
    ref = oracle.token_attention_backward(S.cpu().numpy(), c.H, p["Wq"], p["bq"], p["Wk"],
                                          p["bk"], p["Wv"], p["bv"], p["Wo"], p["bo"],
                                          dSp.cpu().numpy())
    for k in ("dS", "dWq", "dbq", "dWk", "dWv", "dbv", "dWo", "dbo"):
        check(k, ga[k], ref[k], "f32")
    check_key_bias(ga["dbk"], ga["dbq"])


@pytest.mark.parametrize("shape", SHAPES, ids=IDS)
def test_deslice(cases, shape):
    say(f"deslice {shape}")
    c, g, (f, _) = get_case(cases, shape)
    Sp = g.torch.from_numpy(f["Sp"].astype(np.float32)).cuda()
    y = g.deslice(Sp)
    check("y", y, oracle.deslice(f["W"], Sp.cpu().numpy()), c.dt)


@pytest.mark.parametrize("shape", SHAPES, ids=IDS)
def test_deslice_backward(cases, shape):
    say(f"deslice_backward {shape}")
    c, g, (f, gr) = get_case(cases, shape)
    dSp = g.deslice_backward()
    check("dSp", dSp, gr["dSp"], c.dt)


@pytest.mark.parametrize("shape", SHAPES, ids=IDS)
def test_token_attention_backward(cases, shape):
    say(f"token_attention_backward {shape}")
    c, g, (f, _) = get_case(cases, shape)
    S = g.torch.from_numpy(f["S"].astype(np.float32)).cuda()
    rng = np.random.default_rng(5)
    dSp = g.torch.from_numpy(rng.standard_normal((c.M, c.C)).astype(np.float32)).cuda()
    ga = g.attention_backward(S, dSp)
    p = oracle_params(c)
    ref = oracle.token_attention_backward(S.cpu().numpy(), c.H, p["Wq"], p.get("bq"), p["Wk"],
                                          p.get("bk"), p["Wv"], p.get("bv"), None, None,
                                          dSp.cpu().numpy())
    for k in ("dS", "dWq", "dbq", "dWk", "dWv", "dbv"):
        check(k, ga[k], ref[k], "f32")
    check_key_bias(ga["dbk"], ga["dbq"])


# heads too large (D = C) or too narrow (D = 2) for the fused per-head
# kernels: the general projection + core kernels
GENERAL_HEADS = [(300, 128, 1, 64, "f32"), (300, 32, 16, 8, "f32")]


@pytest.mark.parametrize("shape", GENERAL_HEADS,
                         ids=[f"C{c}-H{h}-M{m}" for _, c, h, m, _ in GENERAL_HEADS])
def test_token_attention_general_heads(cases, shape):
    say(f"token_attention (general heads) {shape}")
    c, g, (f, _) = get_case(cases, shape)
    S = g.torch.from_numpy(f["S"].astype(np.float32)).cuda()
    p = oracle_params(c)
    check("Sp", g.attention(S), f["Sp"], "f32")
    rng = np.random.default_rng(6)
    dSp = g.torch.from_numpy(rng.standard_normal((c.M, c.C)).astype(np.float32)).cuda()
    ga = g.attention_backward(S, dSp)
    ref = oracle.token_attention_backward(S.cpu().numpy(), c.H, p["Wq"], p.get("bq"), p["Wk"],
                                          p.get("bk"), p["Wv"], p.get("bv"), None, None,
                                          dSp.cpu().numpy())
    for k in ("dS", "dWq", "dbq", "dWk", "dWv", "dbv"):
        check(k, ga[k], ref[k], "f32")
    check_key_bias(ga["dbk"], ga["dbq"])


def _slice_backward_ref(c, f, dS, Sp, use_dY):
    """Oracle of pa_slice_aggregate_backward for the given dS / Sp / dY."""
    p = oracle_params(c)
    dW = np.zeros((c.N, c.M))
    dx = np.zeros((c.N, c.C))
    if dS is not None:
        dx_a, dW_a = oracle.aggregate_backward(c.x, f["W"], f["num"], f["den"], dS, c.eps)
        dx += dx_a
        dW += dW_a
    if use_dY:
        _, dW_d = oracle.deslice_backward(f["W"], Sp, c.dY)
        dW += dW_d
    sw = oracle.slice_weights_backward(c.x, c.G, p["A"], p.get("b"), p.get("a"),
                                       p.get("b_t", 0.0), c.tau0, c.tau_min, dW)
    sw["dx"] = sw["dx"] + dx
    return sw


@pytest.mark.parametrize("terms", ["both", "states", "deslice"])
@pytest.mark.parametrize("shape", SHAPES, ids=IDS)
def test_slice_aggregate_backward(cases, shape, terms):
    say(f"slice_aggregate_backward {shape} {terms}")
    c, g, (f, gr) = get_case(cases, shape)
    use_dS = terms in ("both", "states")
    use_dY = terms in ("both", "deslice")
    # the forward quantities, as fp32, are the inputs of both sides
    f32 = lambda a: g.torch.from_numpy(np.asarray(a, dtype=np.float32)).cuda()
    num, den, Sp = f32(f["num"]), f32(f["den"]), f32(f["Sp"])
    dS = f32(gr["dS"]) if use_dS else None
    out = g.slice_backward(num, den, dS, Sp if use_dY else None, use_dY=use_dY)
    f64 = dict(f)
    f64["num"], f64["den"] = host(num), host(den)
    ref = _slice_backward_ref(c, f64, host(dS) if use_dS else None, host(Sp), use_dY)
    for k in ("dx", "dA", "db", "da"):
        check(k, out[k], ref[k], c.dt)
    check_ada_temp(out, ref, c.dt)
    assert host(out["dtau0"])[0] == host(out["db_t"])[0]


@pytest.mark.parametrize("shape", SHAPES, ids=IDS)
def test_slice_weights_backward(cases, shape):
    say(f"slice_weights_backward {shape}")
    c, g, (f, _) = get_case(cases, shape)
    rng = np.random.default_rng(9)
    dW = rng.standard_normal((c.N, c.M)).astype(np.float32)
    dtau = rng.standard_normal(c.N).astype(np.float32)
    t = lambda a: g.torch.from_numpy(a).cuda()
    out = g.weights_backward(t(dW), t(dtau))
    p = oracle_params(c)
    ref = oracle.slice_weights_backward(c.x, c.G, p["A"], p.get("b"), p.get("a"),
                                        p.get("b_t", 0.0), c.tau0, c.tau_min, dW, dtau)
    for k in ("dx", "dA", "db", "da"):
        check(k, out[k], ref[k], c.dt)
    check_ada_temp(out, ref, c.dt)


# The chain feeds every call the previous calls' outputs instead of the
# oracle's, through the ABI's fp32 token tensors.  Those roundings alone use
# under half of the fp32 bar (tests/test_oracle_rounding.py, on the oracle),
# so the chained layer is held to the per-call bars.
CHAIN_TOL = TOL


@pytest.mark.parametrize("shape", SHAPES, ids=IDS)
def test_layer_chain(cases, shape):
    """Forward then backward of the whole layer, GPU outputs feeding GPU calls."""
    say(f"layer {shape}")
    c, g, (f, gr) = get_case(cases, shape)
    out = g.layer()
    for k in ("num", "den", "S", "Sp", "y"):
        check(k, out[k], f[k], c.dt, CHAIN_TOL[c.dt])
    for k in ("dSp", "dS", "dWq", "dbq", "dWk", "dWv", "dbv", "dx", "dA", "db", "da"):
        check(k, out[k], gr[k], c.dt, CHAIN_TOL[c.dt])
    check_ada_temp(out, gr, c.dt, CHAIN_TOL[c.dt])
    check_key_bias(out["dbk"], out["dbq"], c.dt)


@pytest.mark.parametrize("shape", [(3001, 256, 8, 32, "bf16"), (50003, 256, 8, 64, "bf16")],
                         ids=["per-wave", "cooperative"])
def test_deterministic(cases, shape):
    """Two runs of the layer are bitwise identical (every sum in a fixed
    order; the second shape runs the cooperative slice backward)."""
    c, g, _ = get_case(cases, shape)
    a = g.layer()
    b = g.layer()
    for k in a:
        assert g.torch.equal(a[k], b[k]), k


@pytest.mark.parametrize("shape", SHAPES, ids=IDS)
def test_slice_aggregate_w(cases, shape):
    """The stored-weights aggregate: num, den, S bitwise those of
    pa_slice_aggregate (same contraction), and W the oracle's weights
    (Eq. 3, 4) rounded to the storage dtype."""
    say(f"slice_aggregate_w {shape}")
    c, g, (f, _) = get_case(cases, shape)
    num, den, S = g.aggregate()
    num_w, den_w, S_w, W = g.aggregate_w()
    for k, a, b in (("num", num, num_w), ("den", den, den_w), ("S", S, S_w)):
        assert g.torch.equal(a, b), k
    check("W", W, f["W"], c.dt)
    check("num", num_w, f["num"], c.dt)


@pytest.mark.parametrize("shape", SHAPES, ids=IDS)
def test_deslice_w(cases, shape):
    say(f"deslice_w {shape}")
    c, g, (f, _) = get_case(cases, shape)
    W = dev(f["W"].astype(np.float32), c.dt)  # the oracle's weights, in the storage dtype
    Sp = dev(f["Sp"].astype(np.float32))
    y = g.deslice_w(W, Sp)
    check("y", y, oracle.deslice(host(W), host(Sp)), c.dt)


@pytest.mark.parametrize("shape", SHAPES, ids=IDS)
def test_deslice_backward_w(cases, shape):
    say(f"deslice_backward_w {shape}")
    c, g, (f, _) = get_case(cases, shape)
    W = dev(f["W"].astype(np.float32), c.dt)
    dSp = g.deslice_backward_w(W)
    check("dSp", dSp, oracle.deslice_backward(host(W), f["Sp"], c.dY)[0], c.dt)


@pytest.mark.parametrize("shape", SHAPES, ids=IDS)
def test_layer_chain_w(cases, shape):
    """The whole layer with stored weights, GPU outputs feeding GPU calls."""
    say(f"layer_w {shape}")
    c, g, (f, gr) = get_case(cases, shape)
    out = g.layer_w()
    for k in ("num", "den", "S", "Sp", "y"):
        check(k, out[k], f[k], c.dt, CHAIN_TOL[c.dt])
    for k in ("dSp", "dS", "dWq", "dbq", "dWk", "dWv", "dbv", "dx", "dA", "db", "da"):
        check(k, out[k], gr[k], c.dt, CHAIN_TOL[c.dt])
    check_ada_temp(out, gr, c.dt, CHAIN_TOL[c.dt])


def test_kernel_timing_hook(cases):
    """pa_time_kernel brackets exactly one streaming kernel per call with the
    caller's events and changes no output."""
    from paper_2502_02414_amd import binding as B
    shape = (66013, 256, 8, 32, "bf16")
    c, g, _ = get_case(cases, shape)
    a, aw = g.layer(), g.layer_w()
    for call in ("pa_slice_aggregate", "pa_deslice", "pa_deslice_backward",
                 "pa_slice_aggregate_backward", "pa_slice_aggregate_w", "pa_deslice_w",
                 "pa_deslice_backward_w"):
        e0, e1, c0, c1 = B.HipEvent(), B.HipEvent(), B.HipEvent(), B.HipEvent()
        B.pa_time_kernel(call, e0, e1)
        run = g.layer_w if call.endswith("_w") else g.layer
        ref = aw if call.endswith("_w") else a
        try:
            c0.record()
            b = run()
            c1.record()
            g.torch.cuda.synchronize()
        finally:
            B.pa_time_kernel(None)
        kernel_ms, layer_ms = e0.elapsed_ms(e1), c0.elapsed_ms(c1)
        say(f"  {call}: kernel {kernel_ms * 1e3:.1f} us of a {layer_ms * 1e3:.1f} us layer")
        assert 0.0 < kernel_ms < layer_ms
        for k in ref:
            assert g.torch.equal(ref[k], b[k]), (call, k)


@pytest.mark.parametrize("variant", ["no_noise", "no_adatemp", "single_point", "empty_slice",
                                     "no_noise_coop", "no_adatemp_coop", "single_point_coop",
                                     "empty_slice_coop"])
def test_edge_cases(variant):
    """No noise, no Ada-Temp (constant temperature), a single point and an
    empty slice; the *_coop variants run them at bf16 rows of 256 channels
    with 40 to 64 slices, the cooperative slice backward's shapes."""
    say(f"edge {variant}")
    if variant == "no_noise":
        c = make_case(300, 64, 4, 16, "f32", noise=False)
    elif variant == "no_adatemp":
        c = make_case(300, 64, 4, 16, "bf16", ada=False)
    elif variant == "single_point":
        c = make_case(1, 32, 1, 3, "f32")
    elif variant == "no_noise_coop":
        c = make_case(3001, 256, 8, 64, "bf16", noise=False)
    elif variant == "no_adatemp_coop":
        c = make_case(2003, 256, 8, 40, "bf16", ada=False)
    elif variant == "single_point_coop":
        c = make_case(1, 256, 8, 64, "bf16")
    else:
        coop = variant == "empty_slice_coop"
        c = make_case(2000, 256, 8, 64, "bf16") if coop else make_case(500, 64, 4, 8, "f32")
        c.p["b"] = c.p["b"].copy()
        c.p["b"][2] = -60.0            # slice 2 is (numerically) empty: den < eps
        c.p["A"] = c.p["A"].copy()
        c.p["A"][:, 2] = 0.0
    g = Gpu(c)
    f, gr = oracle_layer(c)
    if variant.startswith("empty_slice"):
        assert f["den"][2] < c.eps
    for out in (g.layer(), g.layer_w()):  # recomputed, then stored weights
        for k in ("num", "den", "S", "Sp", "y"):
            check(k, out[k], f[k], c.dt)
        for k in ("dSp", "dS", "dx", "dA", "db", "da"):
            check(k, out[k], gr[k], c.dt)


@pytest.mark.parametrize("name", ["grid2d_16k_f32", "ellipsoid_32k_bf16"])
def test_workload_inputs(name):
    """The benchmark workloads' own inputs (their geometry, seeds and zero
    biases), the whole layer chained, recomputed and with stored weights."""
    from paper_2502_02414_amd import inputs as I
    w = I.WORKLOADS[name]
    say(f"workload {name}")
    c = make_case(w.N, w.C, w.H, w.M, w.dtype, workload=w, biases=False)
    g = Gpu(c)
    f, gr = oracle_layer(c)
    for out in (g.layer(), g.layer_w()):
        for k in ("num", "den", "S", "Sp", "y"):
            check(k, out[k], f[k], c.dt)
        for k in ("dSp", "dS", "dWq", "dbq", "dWk", "dWv", "dbv", "dx", "dA", "db", "da"):
            check(k, out[k], gr[k], c.dt)
        check_ada_temp(out, gr, c.dt)
        check_key_bias(out["dbk"], out["dbq"], c.dt)

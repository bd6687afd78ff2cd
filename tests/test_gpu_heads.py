"""Per-head slicing on the GPU vs the CPU oracle, through the C ABI.

The layout calls are checked bit for bit (the relayout) or against float64
host sums (the expansion and sum over heads).  The per-head layer
(paper_2502_02414_amd.heads: the layer's streaming calls per head on the
head-major x, one H-head token attention with block-diagonal shared
projections) is compared with ``oracle.heads_layer_forward`` /
``heads_layer_backward`` on the same seeded inputs, every output tensor by
relative L2 against the per-dtype bar: sizes of several tiles with a ragged
tail, per-head and shared slice parameters, with and without the output
projection, and the Transolver mode (no noise, constant temperature); and
at the million-point car workload's full size with per-head slicing.
"""
import numpy as np
import pytest

import oracle
from paper_2502_02414_amd import binding as B
from paper_2502_02414_amd import inputs as I
from pa_cases import TOL, dev, host, rel_l2, say

pytestmark = pytest.mark.gpu


def check(name, got, ref, dt):
    e = rel_l2(got, ref)
    say(f"  {name:8s} rel_l2 = {e:.3e}  (bar {TOL[dt]:.0e})")
    assert np.isfinite(e) and e <= TOL[dt], (name, e)


@pytest.mark.parametrize("dt,R,H,D", [("bf16", 1001, 4, 32), ("bf16", 77, 8, 8),
                                       ("f32", 999, 3, 4), ("f32", 64, 2, 128)])
def test_heads_relayout_exact(dt, R, H, D):
    import torch
    say(f"relayout {dt} R={R} H={H} D={D}")
    x = I.normal(3, 9, 0, R * H * D, dtype=np.float32).reshape(R, H * D)
    if dt == "bf16":
        x = I.round_bf16(x)
    xd = dev(x, dt)
    xh = torch.empty(H, R, D, dtype=xd.dtype, device="cuda")
    B.pa_heads_relayout(xd, xh, H, to_heads=True)
    back = torch.empty_like(xd)
    B.pa_heads_relayout(xh, back, H, to_heads=False)
    torch.cuda.synchronize()
    want = x.reshape(R, H, D).transpose(1, 0, 2)
    np.testing.assert_array_equal(host(xh), want)
    assert torch.equal(back, xd)


@pytest.mark.parametrize("H,D", [(8, 32), (4, 64), (3, 5)])
def test_heads_expand_and_sum(H, D):
    import torch
    say(f"expand/sum H={H} D={D}")
    W = I.normal(5, 9, 0, D * D, dtype=np.float32).reshape(D, D)
    v = I.normal(5, 10, 0, D, dtype=np.float32)
    Wd, vd = dev(W), dev(v)
    bd = torch.empty(H * D, H * D, dtype=torch.float32, device="cuda")
    B.pa_heads_expand(Wd, bd, H, blockdiag=True)
    tile = torch.empty(H * D, dtype=torch.float32, device="cuda")
    B.pa_heads_expand(vd, tile, H, blockdiag=False)
    np.testing.assert_array_equal(host(bd), np.kron(np.eye(H), W))
    np.testing.assert_array_equal(host(tile), np.tile(v, H))
    # sums over the heads: diagonal blocks of a full matrix, rows of [H, L]
    F = I.normal(5, 11, 0, (H * D) ** 2, dtype=np.float32).reshape(H * D, H * D)
    P = I.normal(5, 12, 0, H * 3 * D, dtype=np.float32).reshape(H, 3 * D)
    s_bd = torch.empty(D, D, dtype=torch.float32, device="cuda")
    B.pa_heads_sum(dev(F), s_bd, H, blockdiag=True)
    s_v = torch.empty(3 * D, dtype=torch.float32, device="cuda")
    B.pa_heads_sum(dev(P), s_v, H, blockdiag=False)
    want_bd = sum(F[h * D:(h + 1) * D, h * D:(h + 1) * D].astype(np.float64) for h in range(H))
    np.testing.assert_allclose(host(s_bd), want_bd, rtol=1e-7, atol=1e-7)
    np.testing.assert_allclose(host(s_v), P.astype(np.float64).sum(axis=0), rtol=1e-7, atol=1e-7)
    # the same sums (and a scalar's) in one batched launch: the same bits
    S1 = I.normal(5, 13, 0, H, dtype=np.float32)
    b_bd = torch.empty(D, D, dtype=torch.float32, device="cuda")
    b_v = torch.empty(3 * D, dtype=torch.float32, device="cuda")
    b_s = torch.empty(1, dtype=torch.float32, device="cuda")
    s_s = torch.empty(1, dtype=torch.float32, device="cuda")
    B.pa_heads_sum(dev(S1), s_s, H, blockdiag=False)
    B.pa_heads_sum_batch([(dev(F), b_bd, True), (dev(P), b_v, False), (dev(S1), b_s, False)], H)
    for got, want in ((b_bd, s_bd), (b_v, s_v), (b_s, s_s)):
        np.testing.assert_array_equal(host(got), host(want))


def head_case(N, H, D, M, dt, shared, noise, out_proj, geometry="normal", seed=31, w=None):
    w = w or I.small("heads", N, H * D, H, M, dt, geometry=geometry, seed=seed)
    x = I.make_x(w, N)
    G = I.make_head_gumbel(w, N) if noise else None
    p = I.make_head_params(w, shared=shared, biases=True, out_proj=out_proj)
    if not noise:
        p["a"] = None                      # Transolver mode: constant temperature
    dY = I.make_grad(w, N)
    return w, x, G, p, dY


def run_gpu(w, N, x, G, p, dY, dt, streams=2, batched=None):
    import torch
    from paper_2502_02414_amd.heads import HeadSlicedLayer
    H, D, M = w.H, w.C // w.H, w.M
    pd = {}
    for k, v in p.items():
        if v is None:
            continue
        if k == "b_t":
            pd[k] = float(v) if np.ndim(v) == 0 else [float(t) for t in v]
        elif k in ("A", "a"):
            pd[k] = dev(v, dt)
        else:
            pd[k] = dev(v)
    L = HeadSlicedLayer(N, H, D, M, pd, torch.bfloat16 if dt == "bf16" else torch.float32,
                        w.tau0, w.tau_min, w.eps, streams=streams, batched=batched)
    xh = L.to_heads(dev(x, dt))
    Gd = dev(G, dt) if G is not None else None
    y = L.from_heads(L.forward(xh, Gd))
    dxh, g = L.backward(L.to_heads(dev(dY, dt)))
    dx = L.from_heads(dxh)
    torch.cuda.synchronize()
    out = {"y": host(y), "dx": host(dx)}
    out.update({k: host(v) for k, v in g.items()})
    return out


def compare(w, x, G, p, dY, out, dt):
    f = oracle.heads_layer_forward(x, G, p, w.tau0, w.tau_min, w.eps, w.H)
    g = oracle.heads_layer_backward(x, G, p, w.tau0, w.tau_min, w.eps, w.H, f, dY)
    check("y", out["y"], f["y"], dt)
    check("dx", out["dx"], g["dx"], dt)
    # with one point every slice's state is that point: a head's tokens are
    # equal, its attention is uniform and its outputs are equal, so y does
    # not depend on the slice weights; the query, key and slice-parameter
    # gradients are exactly zero (nothing to compare but rounding)
    one = x.shape[0] == 1
    qk = () if one else ("dWq", "dbq", "dWk")
    for k in qk + ("dWv", "dbv", "dWo", "dbo") + (() if one else ("dA", "db")):
        if k in g and p.get(k[1:]) is not None:
            check(k, out[k], g[k], dt)
    if qk:
        # the key bias moves every logit of a query by the same amount, so
        # its gradient is zero in exact arithmetic: only rounding is left
        scale = np.abs(g["dbq"]).max()
        assert np.abs(out["dbk"]).max() <= TOL[dt] * scale, (np.abs(out["dbk"]).max(), scale)
    # db_t alone is a sum over the points of terms of both signs (a small
    # fraction of the sum of their magnitudes), so it is checked with the
    # other parameters of its Linear: (a, b_t) with Ada-Temp; with a constant
    # temperature, (b, b_t), the biases of the logits and the temperature
    if one:
        pass
    elif p.get("a") is not None:
        da = np.concatenate([out["da"].ravel(), out["db_t"].ravel()])
        check("d(a,b_t)", da, np.concatenate([np.ravel(g["da"]), np.ravel(g["db_t"])]), dt)
        # d tau0 sums the heads' d b_t, which can cancel (by a factor of ~80
        # at H = 4, D = 48): its error is bounded by the bar times the
        # magnitude of the terms it adds
        ref = float(np.ravel(g["dtau0"])[0])
        scale = max(abs(ref), float(np.abs(np.ravel(g["db_t"])).sum()))
        err = abs(float(out["dtau0"].ravel()[0]) - ref)
        say(f"  dtau0    |err| = {err:.3e}  (bar {TOL[dt]:.0e} x {scale:.3e})")
        assert err <= TOL[dt] * scale, ("dtau0", err, scale)
    else:
        db = np.concatenate([out["db"].ravel(), out["db_t"].ravel()])
        check("d(b,b_t)", db, np.concatenate([np.ravel(g["db"]), np.ravel(g["db_t"])]), dt)
    # d tau0 is the sum of the heads' d b_t
    np.testing.assert_allclose(out["dtau0"].ravel(), [np.sum(out["db_t"], dtype=np.float64)],
                               rtol=1e-6, atol=0)


CASES = [
    # dt, N, H, D, M, shared, noise, out_proj
    ("f32", 3000, 4, 32, 16, False, True, False),
    ("f32", 2049, 2, 64, 32, True, True, True),
    ("f32", 1500, 4, 32, 8, False, False, False),
    ("bf16", 20000, 8, 32, 32, False, True, True),
    ("bf16", 9001, 4, 64, 64, False, True, False),
    ("bf16", 5000, 2, 128, 16, True, False, False),
    ("f32", 1000, 2, 32, 12, False, True, False),   # M not a multiple of 8: one call per head
    ("f32", 1, 2, 32, 8, False, True, True),          # one point
    ("bf16", 17, 4, 64, 16, True, True, False),       # one tile and a ragged tail
    # head widths between the kernels' widths (D = 48, 16, 80)
    ("bf16", 3001, 4, 48, 32, False, True, True),
    ("f32", 2000, 3, 16, 24, False, True, False),
    ("bf16", 1500, 2, 80, 16, True, True, False),
]


@pytest.mark.parametrize("dt,N,H,D,M,shared,noise,out_proj", CASES)
def test_heads_layer_parity(dt, N, H, D, M, shared, noise, out_proj):
    say(f"heads layer {dt} N={N} H={H} D={D} M={M} shared={shared} noise={noise} "
        f"out_proj={out_proj}")
    w, x, G, p, dY = head_case(N, H, D, M, dt, shared, noise, out_proj)
    out = run_gpu(w, N, x, G, p, dY, dt)
    compare(w, x, G, p, dY, out, dt)


@pytest.mark.parametrize("shared", [False, True])
def test_heads_launch_modes_bitwise_identical(shared):
    """All heads in one launch per kernel (pa_heads_*), and one call per head
    on 1, 2 or 3 streams: every head's arithmetic and summation order is the
    same, so every mode gives the same bits."""
    say(f"heads layer batched vs per-head calls: bf16 N=20000 H=8 D=32 M=32 shared={shared}")
    w, x, G, p, dY = head_case(20000, 8, 32, 32, "bf16", shared, True, True)
    outs = [run_gpu(w, 20000, x, G, p, dY, "bf16", batched=True)]
    outs += [run_gpu(w, 20000, x, G, p, dY, "bf16", streams=k, batched=False) for k in (1, 2, 3)]
    for o in outs[1:]:
        for k, v in outs[0].items():
            np.testing.assert_array_equal(o[k], v, err_msg=k)


def test_heads_layer_full_size_car():
    """Per-head slicing at the million-point car workload's shape: N = 1M,
    C = 256 as H = 8 heads of D = 32, M = 32 slices per head, bf16."""
    w = I.WORKLOADS["car_1m_bf16"]
    say(f"heads full size {w.name}: N={w.N} H={w.H} D={w.C // w.H} M={w.M} {w.dtype}")
    w, x, G, p, dY = head_case(w.N, w.H, w.C // w.H, w.M, w.dtype, False, True, False, w=w)
    out = run_gpu(w, w.N, x, G, p, dY, w.dtype)
    say("  gpu done; oracle forward + backward ...")
    compare(w, x, G, p, dY, out, w.dtype)

"""Two more pins of the oracle's layer, each written here from the
equations, independently of the oracle's C code:

* the forward at small sizes (N <= 64 points; (C, H, M) in {(16, 1, 1),
  (32, 2, 4), (64, 4, 16)}) against an explicit per-element evaluation in
  plain Python float64 loops: slice logits and Ada-Temp (Eq. 3, Eq. 4),
  the Gumbel-softmax over the slices (Eq. 4), the weight-normalised states
  (Eq. 1), multi-head attention among the states (Eq. 2) and the deslice
  (Section 3, the text after Eq. 2);
* the backward against torch's float64 autograd of the same forward
  written with torch tensor operations (plain, with points clamped at the
  temperature floor, with a slice whose denominator is floored, and
  without the output projection).
"""
import math

import numpy as np
import pytest

import oracle


def _case(N, C, H, M, seed, out_proj=True, clamp=False, empty=False):
    rng = np.random.default_rng(seed)
    r = lambda *s, sc=1.0: sc * rng.standard_normal(s)
    x, G = r(N, C), r(N, M)
    p = {"A": r(C, M, sc=0.6), "b": r(M, sc=0.3), "a": r(C, sc=0.15), "b_t": 0.05,
         "Wq": r(C, C, sc=0.3), "bq": r(C, sc=0.1), "Wk": r(C, C, sc=0.3), "bk": r(C, sc=0.1),
         "Wv": r(C, C, sc=0.3), "bv": r(C, sc=0.1)}
    if out_proj:
        p["Wo"], p["bo"] = r(C, C, sc=0.3), r(C, sc=0.1)
    tau0 = 0.2 if clamp else 0.9
    if empty and M > 1:
        p["b"][M - 1] = -60.0  # that slice's weights ~ e^-60: den below eps
        p["A"][:, M - 1] = 0.0
    dY = r(N, C)
    return x, G, p, tau0, dY


def _explicit_forward(x, G, p, tau0, tau_min, eps, H):
    """Eq. 1-4 element by element (Python floats)."""
    N, C = x.shape
    M = G.shape[1]
    D = C // H
    W = [[0.0] * M for _ in range(N)]
    for i in range(N):
        t = tau0 + p["b_t"] + sum(x[i, c] * p["a"][c] for c in range(C))
        tau = max(t, tau_min)
        z = [(p["b"][j] + sum(x[i, c] * p["A"][c, j] for c in range(C)) + G[i, j]) / tau
             for j in range(M)]
        m = max(z)
        e = [math.exp(v - m) for v in z]
        s = sum(e)
        W[i] = [v / s for v in e]
    den = [sum(W[i][j] for i in range(N)) for j in range(M)]
    S = [[sum(W[i][j] * x[i, c] for i in range(N)) / max(den[j], eps) for c in range(C)]
         for j in range(M)]

    def lin(X, Wm, b):
        return [[b[o] + sum(X[j][k] * Wm[k, o] for k in range(len(X[j])))
                 for o in range(Wm.shape[1])] for j in range(len(X))]

    Q, K, V = lin(S, p["Wq"], p["bq"]), lin(S, p["Wk"], p["bk"]), lin(S, p["Wv"], p["bv"])
    O = [[0.0] * C for _ in range(M)]
    for h in range(H):
        cols = range(h * D, (h + 1) * D)
        for q in range(M):
            sc = [sum(Q[q][c] * K[k][c] for c in cols) / math.sqrt(D) for k in range(M)]
            m = max(sc)
            e = [math.exp(v - m) for v in sc]
            s = sum(e)
            for c in cols:
                O[q][c] = sum(e[k] / s * V[k][c] for k in range(M))
    Sp = lin(O, p["Wo"], p["bo"]) if "Wo" in p else O
    y = [[sum(W[i][j] * Sp[j][c] for j in range(M)) for c in range(C)] for i in range(N)]
    return {"W": np.array(W), "S": np.array(S), "Sp": np.array(Sp), "y": np.array(y)}


@pytest.mark.parametrize("shape", [(40, 16, 1, 1), (48, 32, 2, 4), (64, 64, 4, 16)],
                         ids=lambda s: "N{}-C{}-H{}-M{}".format(*s))
def test_forward_matches_explicit_evaluation(shape):
    N, C, H, M = shape
    x, G, p, tau0, _ = _case(N, C, H, M, seed=N + C)
    f = oracle.layer_forward(x, G, p, tau0, 0.05, 1e-5, H)
    ref = _explicit_forward(x, G, p, tau0, 0.05, 1e-5, H)
    for k, v in ref.items():
        err = np.abs(np.asarray(f[k]) - v).max() / max(np.abs(v).max(), 1e-300)
        assert err <= 1e-12, (k, err)


def _torch_loss(x, G, p, tau0, tau_min, eps, H, dY):
    import torch
    t = tau0 + p["b_t"] + x @ p["a"]
    tau = torch.clamp(t, min=tau_min)
    z = (x @ p["A"] + p["b"] + G) / tau[:, None]
    W = torch.softmax(z, dim=1)
    den = W.sum(0)
    S = (W.T @ x) / torch.clamp(den, min=eps)[:, None]
    Q, K, V = S @ p["Wq"] + p["bq"], S @ p["Wk"] + p["bk"], S @ p["Wv"] + p["bv"]
    M, C = S.shape
    D = C // H
    heads = []
    for h in range(H):
        sl = slice(h * D, (h + 1) * D)
        P = torch.softmax(Q[:, sl] @ K[:, sl].T / math.sqrt(D), dim=1)
        heads.append(P @ V[:, sl])
    O = torch.cat(heads, dim=1)
    Sp = O @ p["Wo"] + p["bo"] if "Wo" in p else O
    y = W @ Sp
    return (y * dY).sum()


@pytest.mark.parametrize("case", ["plain", "clamped", "empty_slice", "no_out_proj"])
def test_backward_matches_autograd(case):
    import torch
    N, C, H, M, tau_min, eps = 30, 16, 2, 6, 0.05, 1e-5
    x, G, p, tau0, dY = _case(N, C, H, M, seed=3 + len(case), out_proj=case != "no_out_proj",
                              clamp=case == "clamped", empty=case == "empty_slice")
    f = oracle.layer_forward(x, G, p, tau0, tau_min, eps, H)
    if case == "clamped":
        assert (f["t"] < tau_min).any() and (f["t"] > tau_min).any()
    if case == "empty_slice":
        assert f["den"][M - 1] < eps
    g = oracle.layer_backward(x, G, p, tau0, tau_min, eps, H, f, dY)

    T = lambda a: torch.tensor(np.asarray(a, dtype=np.float64), requires_grad=True)
    tx, tG, tdY = T(x), torch.tensor(G), torch.tensor(dY)
    tp = {k: T(v) for k, v in p.items()}
    ttau0 = T(tau0)
    loss = _torch_loss(tx, tG, tp, ttau0, tau_min, eps, H, tdY)
    loss.backward()
    pairs = [("dx", tx.grad), ("dA", tp["A"].grad), ("db", tp["b"].grad),
             ("da", tp["a"].grad), ("db_t", tp["b_t"].grad), ("dtau0", ttau0.grad),
             ("dWq", tp["Wq"].grad), ("dbq", tp["bq"].grad), ("dWk", tp["Wk"].grad),
             ("dbk", tp["bk"].grad), ("dWv", tp["Wv"].grad), ("dbv", tp["bv"].grad)]
    if "Wo" in p:
        pairs += [("dWo", tp["Wo"].grad), ("dbo", tp["bo"].grad)]
    for name, ref in pairs:
        ref = ref.numpy()
        got = np.asarray(g[name], dtype=np.float64).reshape(ref.shape)
        scale = max(np.abs(ref).max(), 1e-12)
        err = np.abs(got - ref).max() / scale
        # dbk is exactly zero in exact arithmetic (a key bias shifts a whole
        # score row): both sides are rounding noise, compared absolutely
        bar = 1e-9 if name != "dbk" else 1e-9 / scale * np.abs(g["dbq"]).max()
        assert err <= bar, (name, err)

"""Python access to the Physics-Attention oracle (plain C, double precision).

TEST INFRASTRUCTURE ONLY.  Only the tests, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import this package.  It shares no
code with the HIP path: it neither imports nor is imported by
``paper_2502_02414_amd``.

Every function takes numpy arrays (any float dtype; upcast exactly to
float64) and returns float64 arrays.  The maths and the readings of the paper
are documented in ``pa_oracle.h``; each wrapper names the passage it follows.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from .build import LIB, build, lib_path

_lib = None
# The library variant this process loads (oracle/build.py): PA_ORACLE_VARIANT
# in the environment, else the portable build; use_variant() before the
# first call chooses another.
_variant = os.environ.get("PA_ORACLE_VARIANT", "portable")


def use_variant(variant: str, rebuild: bool = False) -> str:
    """Load the given library variant from now on (before any oracle call);
    with rebuild, compile it first on this host."""
    global _variant
    if _lib is not None and variant != _variant:
        raise RuntimeError(f"oracle library {_variant} already loaded")
    _variant = variant
    if rebuild or not os.path.exists(lib_path(variant)):
        build(variant=variant)
    return lib_path(variant)


def variant() -> str:
    return _variant


def _load():
    global _lib
    if _lib is None:
        path = lib_path(_variant)
        if not os.path.exists(path):
            build(variant=_variant)
        lib = ctypes.CDLL(path)
        P = ctypes.c_void_p
        I64, I32, D = ctypes.c_int64, ctypes.c_int, ctypes.c_double
        lib.pao_slice_weights.argtypes = [I64, I32, I32, D, D, P, P, P, P, P, D, P, P, P]
        lib.pao_aggregate.argtypes = [I64, I32, I32, D, P, P, P, P, P]
        lib.pao_token_attention.argtypes = [I32, I32, I32, P] + [P] * 8 + [P]
        lib.pao_deslice.argtypes = [I64, I32, I32, P, P, P]
        lib.pao_deslice_backward.argtypes = [I64, I32, I32, P, P, P, P, P]
        lib.pao_token_attention_backward.argtypes = [I32, I32, I32, P] + [P] * 8 + [P, P] + [P] * 8
        lib.pao_aggregate_backward.argtypes = [I64, I32, I32, D, P, P, P, P, P, P, P]
        lib.pao_slice_weights_backward.argtypes = (
            [I64, I32, I32, D, D, P, P, P, P, P, D, P, P, P, P, P, P, P, P])
        lib.pao_layernorm.argtypes = [I64, I32, D, P, P, P, P, P, P]
        lib.pao_layernorm_backward.argtypes = [I64, I32, D, P, P, P, P, P, P]
        lib.pao_gelu.argtypes = [I64, P, P]
        lib.pao_gelu_backward.argtypes = [I64, P, P, P]
        lib.pao_shard_points.restype = I32
        lib.pao_num_threads.restype = I32
        lib.pao_set_num_threads.argtypes = [I32]
        _lib = lib
    return _lib


def _in(a):
    """float64 C-contiguous copy (exact upcast) or None."""
    if a is None:
        return None
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def num_threads() -> int:
    return int(_load().pao_num_threads())


def set_num_threads(n: int) -> None:
    _load().pao_set_num_threads(int(n))


def shard_points() -> int:
    return int(_load().pao_shard_points())


def slice_weights(x, G, A, b, a, b_t, tau0, tau_min):
    """Eq. 3 (Ada-Temp) and Eq. 4 (Rep-Slice).  Returns (W [N,M], tau [N], t [N])."""
    x, G, A, b, a = map(_in, (x, G, A, b, a))
    N, C = x.shape
    M = A.shape[1]
    W = np.empty((N, M))
    tau = np.empty(N)
    t = np.empty(N)
    _load().pao_slice_weights(N, C, M, float(tau0), float(tau_min), _p(x), _p(G), _p(A),
                              _p(b), _p(a), float(b_t), _p(W), _p(tau), _p(t))
    return W, tau, t


def aggregate(x, W, eps):
    """Eq. 1 states, sharded as in Section 4.2.  Returns (num [M,C], den [M], S [M,C])."""
    x, W = _in(x), _in(W)
    N, C = x.shape
    M = W.shape[1]
    num = np.empty((M, C))
    den = np.empty(M)
    S = np.empty((M, C))
    _load().pao_aggregate(N, C, M, float(eps), _p(x), _p(W), _p(num), _p(den), _p(S))
    return num, den, S


def token_attention(S, H, Wq, bq, Wk, bk, Wv, bv, Wo=None, bo=None):
    """Eq. 2 with H heads of D = C/H channels.  Returns Sp [M,C]."""
    S, Wq, bq, Wk, bk, Wv, bv, Wo, bo = map(_in, (S, Wq, bq, Wk, bk, Wv, bv, Wo, bo))
    M, C = S.shape
    Sp = np.empty((M, C))
    _load().pao_token_attention(M, C, int(H), _p(S), _p(Wq), _p(bq), _p(Wk), _p(bk),
                                _p(Wv), _p(bv), _p(Wo), _p(bo), _p(Sp))
    return Sp


def deslice(W, Sp):
    """Deslice (Section 3): y = W Sp.  Returns y [N,C]."""
    W, Sp = _in(W), _in(Sp)
    N, M = W.shape
    C = Sp.shape[1]
    y = np.empty((N, C))
    _load().pao_deslice(N, C, M, _p(W), _p(Sp), _p(y))
    return y


def deslice_backward(W, Sp, dY):
    """Chain rule of the deslice.  Returns (dSp [M,C], dW [N,M])."""
    W, Sp, dY = map(_in, (W, Sp, dY))
    N, M = W.shape
    C = Sp.shape[1]
    dSp = np.empty((M, C))
    dW = np.empty((N, M))
    _load().pao_deslice_backward(N, C, M, _p(W), _p(Sp), _p(dY), _p(dSp), _p(dW))
    return dSp, dW


def token_attention_backward(S, H, Wq, bq, Wk, bk, Wv, bv, Wo, bo, dSp):
    """Chain rule of Eq. 2.  Returns dict with dS and the parameter gradients."""
    S, Wq, bq, Wk, bk, Wv, bv, Wo, bo, dSp = map(
        _in, (S, Wq, bq, Wk, bk, Wv, bv, Wo, bo, dSp))
    M, C = S.shape
    out = {k: np.empty((C, C)) for k in ("dWq", "dWk", "dWv")}
    out.update({k: np.empty(C) for k in ("dbq", "dbk", "dbv")})
    out["dS"] = np.empty((M, C))
    if Wo is not None:
        out["dWo"] = np.empty((C, C))
        out["dbo"] = np.empty(C)
    _load().pao_token_attention_backward(
        M, C, int(H), _p(S), _p(Wq), _p(bq), _p(Wk), _p(bk), _p(Wv), _p(bv), _p(Wo),
        _p(bo), _p(dSp), _p(out["dS"]), _p(out["dWq"]), _p(out["dbq"]), _p(out["dWk"]),
        _p(out["dbk"]), _p(out["dWv"]), _p(out["dbv"]), _p(out.get("dWo")),
        _p(out.get("dbo")))
    return out


def aggregate_backward(x, W, num, den, dS, eps):
    """Chain rule of Eq. 1.  Returns (dx_direct [N,C], dW [N,M])."""
    x, W, num, den, dS = map(_in, (x, W, num, den, dS))
    N, C = x.shape
    M = W.shape[1]
    dx = np.empty((N, C))
    dW = np.empty((N, M))
    _load().pao_aggregate_backward(N, C, M, float(eps), _p(x), _p(W), _p(num), _p(den),
                                   _p(dS), _p(dx), _p(dW))
    return dx, dW


def slice_weights_backward(x, G, A, b, a, b_t, tau0, tau_min, dW, dtau=None):
    """Chain rule of Eq. 3 + Eq. 4.  Returns dict dx, dA, db, da, db_t, dtau0."""
    x, G, A, b, a, dW, dtau = map(_in, (x, G, A, b, a, dW, dtau))
    N, C = x.shape
    M = A.shape[1]
    out = {"dx": np.empty((N, C)), "dA": np.empty((C, M)), "db": np.empty(M),
           "da": np.empty(C), "db_t": np.empty(1), "dtau0": np.empty(1)}
    _load().pao_slice_weights_backward(
        N, C, M, float(tau0), float(tau_min), _p(x), _p(G), _p(A), _p(b), _p(a),
        float(b_t), _p(dW), _p(dtau), _p(out["dx"]), _p(out["dA"]), _p(out["db"]),
        _p(out["da"]), _p(out["db_t"]), _p(out["dtau0"]))
    out["db_t"] = float(out["db_t"][0])
    out["dtau0"] = float(out["dtau0"][0])
    return out


def layer_forward(x, G, p, tau0, tau_min, eps, H):
    """One Physics-Attention layer forward (Algorithm 1 on one shard).

    ``p`` holds A, b, a, b_t, Wq, bq, Wk, bk, Wv, bv and optionally Wo, bo.
    Returns a dict with W, tau, t, num, den, S, Sp, y.
    """
    W, tau, t = slice_weights(x, G, p["A"], p.get("b"), p.get("a"), p.get("b_t", 0.0),
                              tau0, tau_min)
    num, den, S = aggregate(x, W, eps)
    Sp = token_attention(S, H, p["Wq"], p.get("bq"), p["Wk"], p.get("bk"), p["Wv"],
                         p.get("bv"), p.get("Wo"), p.get("bo"))
    y = deslice(W, Sp)
    return {"W": W, "tau": tau, "t": t, "num": num, "den": den, "S": S, "Sp": Sp, "y": y}


def layer_backward(x, G, p, tau0, tau_min, eps, H, fwd, dY):
    """Chain rule of ``layer_forward`` for the upstream gradient dY [N,C].

    Returns a dict with dSp, dS, dx and every parameter gradient.
    """
    dSp, dW_des = deslice_backward(fwd["W"], fwd["Sp"], dY)
    att = token_attention_backward(fwd["S"], H, p["Wq"], p.get("bq"), p["Wk"], p.get("bk"),
                                   p["Wv"], p.get("bv"), p.get("Wo"), p.get("bo"), dSp)
    dx_agg, dW_agg = aggregate_backward(x, fwd["W"], fwd["num"], fwd["den"], att["dS"], eps)
    sw = slice_weights_backward(x, G, p["A"], p.get("b"), p.get("a"), p.get("b_t", 0.0),
                                tau0, tau_min, dW_des + dW_agg)
    out = dict(att)
    out.update({"dSp": dSp, "dx": dx_agg + sw["dx"], "dA": sw["dA"], "db": sw["db"],
                "da": sw["da"], "db_t": sw["db_t"], "dtau0": sw["dtau0"]})
    return out


# ---------------------------------------------------------------------------
# Block stack: the Transolver++ block around the layer (Section 3: the
# Transformer block with Physics-Attention in place of attention; block
# diagram of Figure 2a), read as pre-norm with residual adds:
#     x1 = x + PA(LN1(x)),   x2 = x1 + MLP(LN2(x1)),
#     MLP(h) = GELU(h W1 + b1) W2 + b2 (GELU(u) = u Phi(u)),
# and PA with Algorithm 1's Project step applied explicitly:
#     x_proj = LN1(x) Wp + bp, then the layer on x_proj (to_out = Wo, bo).
# ---------------------------------------------------------------------------
LN_EPS = 1e-5


def layernorm(x, g, b, eps=LN_EPS):
    """Per-row LayerNorm (biased variance).  Returns (y, mean, rstd)."""
    x, g, b = map(_in, (x, g, b))
    N, C = x.shape
    y, mean, rstd = np.empty((N, C)), np.empty(N), np.empty(N)
    _load().pao_layernorm(N, C, float(eps), _p(x), _p(g), _p(b), _p(y), _p(mean), _p(rstd))
    return y, mean, rstd


def layernorm_backward(x, g, dy, eps=LN_EPS):
    """Chain rule of layernorm.  Returns (dx, dg, db)."""
    x, g, dy = map(_in, (x, g, dy))
    N, C = x.shape
    dx, dg, db = np.empty((N, C)), np.empty(C), np.empty(C)
    _load().pao_layernorm_backward(N, C, float(eps), _p(x), _p(g), _p(dy), _p(dx), _p(dg),
                                   _p(db))
    return dx, dg, db


def gelu(x):
    """GELU x Phi(x), Phi(x) = (1 + erf(x / sqrt 2)) / 2 (standard normal CDF)."""
    x = _in(x)
    y = np.empty_like(x)
    _load().pao_gelu(x.size, _p(x), _p(y))
    return y


def gelu_backward(x, dy):
    x, dy = _in(x), _in(dy)
    dx = np.empty_like(x)
    _load().pao_gelu_backward(x.size, _p(x), _p(dy), _p(dx))
    return dx


def linear(x, W, b=None):
    """y = x W + b: a plain matrix product, numpy's float64 matmul serving as
    the step (a library routine, with no blocking or fusion of our own)."""
    x, W, b = map(_in, (x, W, b))
    y = x @ W
    return y if b is None else y + b


def linear_backward(x, W, dy):
    """Chain rule of linear.  Returns (dx, dW, db) = (dy W^T, x^T dy, 1^T dy)."""
    x, W, dy = map(_in, (x, W, dy))
    return dy @ W.T, x.T @ dy, dy.sum(axis=0)


def block_forward(x, G, p, tau0, tau_min, eps, H, ln_eps=LN_EPS):
    """One block.  ``p`` holds the layer's parameters (A, b, a, b_t, Wq, bq,
    Wk, bk, Wv, bv, optional Wo, bo) plus ln1_g, ln1_b, Wp, bp, ln2_g, ln2_b,
    W1, b1, W2, b2.  Returns (x2, cache)."""
    h, _, _ = layernorm(x, p["ln1_g"], p["ln1_b"], ln_eps)
    xp = linear(h, p["Wp"], p["bp"])
    pa = layer_forward(xp, G, p, tau0, tau_min, eps, H)
    x1 = _in(x) + pa["y"]
    h2, _, _ = layernorm(x1, p["ln2_g"], p["ln2_b"], ln_eps)
    u = linear(h2, p["W1"], p["b1"])
    v = linear(gelu(u), p["W2"], p["b2"])
    x2 = x1 + v
    return x2, {"x": _in(x), "h": h, "xp": xp, "pa": pa, "x1": x1, "h2": h2, "u": u}


def block_backward(dx2, G, p, tau0, tau_min, eps, H, cache, ln_eps=LN_EPS):
    """Chain rule of block_forward.  Returns (dx, grads) with a gradient for
    every parameter of ``p`` (the layer's as in layer_backward)."""
    c = cache
    dx2 = _in(dx2)
    dgu, dW2, db2 = linear_backward(gelu(c["u"]), p["W2"], dx2)
    du = gelu_backward(c["u"], dgu)
    dh2, dW1, db1 = linear_backward(c["h2"], p["W1"], du)
    dx1_ln, dg2, db2n = layernorm_backward(c["x1"], p["ln2_g"], dh2, ln_eps)
    dx1 = dx2 + dx1_ln
    g = layer_backward(c["xp"], G, p, tau0, tau_min, eps, H, c["pa"], dx1)
    dh, dWp, dbp = linear_backward(c["h"], p["Wp"], g["dx"])
    dx_ln, dg1, db1n = layernorm_backward(c["x"], p["ln1_g"], dh, ln_eps)
    grads = {k: v for k, v in g.items() if k not in ("dx", "dSp", "dS")}
    grads.update({"dW2": dW2, "db2": db2, "dW1": dW1, "db1": db1, "dln2_g": dg2,
                  "dln2_b": db2n, "dWp": dWp, "dbp": dbp, "dln1_g": dg1, "dln1_b": db1n})
    return dx1 + dx_ln, grads


def stack_forward(x, Gs, ps, tau0, tau_min, eps, H, ln_eps=LN_EPS):
    """len(ps) blocks in sequence (layer l uses noise Gs[l]).  Returns
    (output, caches)."""
    caches = []
    for G, p in zip(Gs, ps):
        x, cache = block_forward(x, G, p, tau0, tau_min, eps, H, ln_eps)
        caches.append(cache)
    return x, caches


def stack_backward(dy, Gs, ps, tau0, tau_min, eps, H, caches, ln_eps=LN_EPS):
    """Chain rule of stack_forward.  Returns (dx, [grads per layer])."""
    grads = [None] * len(ps)
    for l in reversed(range(len(ps))):
        dy, grads[l] = block_backward(dy, Gs[l], ps[l], tau0, tau_min, eps, H, caches[l], ln_eps)
    return dy, grads



# ---------------------------------------------------------------------------
# Per-head slicing: the heads of Eq. 2 carried into the slicing of Eq. 1.
# The C channels split into H contiguous blocks of D = C/H channels.  Head h
# slices its own block x_h = x[:, hD:(h+1)D] with its own projection A_h
# [D,M], b_h, Ada-Temp a_h, b_t,h and Gumbel noise G_h [N,M] (Eq. 3, Eq. 4),
# forms its own M states S_h [M,D] (Eq. 1), runs one-head attention of width
# D among them with the token projections shared by every head (Eq. 2's
# Linear acting on the last axis of the [H,M,D] states), and its deslice
# W_h S'_h fills the channels hD..(h+1)D of y.  Slice parameters may also be
# shared by every head (A given as [D,M]): then their gradients are the sums
# over the heads.  G is [H,N,M] or None (the Transolver mode has no noise;
# with a None as well the temperature is the constant tau0 + b_t).
# ---------------------------------------------------------------------------
_SLICE_KEYS = ("A", "b", "a", "b_t")
_ATTN_KEYS = ("Wq", "bq", "Wk", "bk", "Wv", "bv", "Wo", "bo")


def _head_params(p, h, shared):
    """The layer parameters of head h: its slice parameters (or the shared
    ones) and the shared token projections."""
    q = {k: p.get(k) for k in _ATTN_KEYS if p.get(k) is not None}
    for k in _SLICE_KEYS:
        v = p.get(k)
        if v is None:
            continue
        if k == "b_t":
            q[k] = float(v) if shared else float(np.asarray(v, dtype=np.float64)[h])
        else:
            q[k] = v if shared else np.asarray(v)[h]
    return q


def heads_shared(p):
    """True when the slice parameters are one set for every head."""
    return np.asarray(p["A"]).ndim == 2


def heads_layer_forward(x, G, p, tau0, tau_min, eps, H):
    """Per-head sliced layer forward on x [N,C].  Returns a dict with y [N,C]
    and "heads", the per-head ``layer_forward`` results (on x_h)."""
    x = _in(x)
    N, C = x.shape
    D = C // H
    assert D * H == C
    shared = heads_shared(p)
    y = np.empty((N, C))
    heads = []
    for h in range(H):
        xh = x[:, h * D:(h + 1) * D]
        f = layer_forward(xh, None if G is None else G[h], _head_params(p, h, shared), tau0,
                          tau_min, eps, 1)
        y[:, h * D:(h + 1) * D] = f["y"]
        heads.append(f)
    return {"y": y, "heads": heads}


def heads_layer_backward(x, G, p, tau0, tau_min, eps, H, fwd, dY):
    """Chain rule of ``heads_layer_forward`` for dY [N,C].  Returns dx [N,C],
    the slice-parameter gradients (per head, stacked on a leading axis of H,
    or summed when the parameters are shared) and the token-projection
    gradients summed over the heads."""
    x, dY = _in(x), _in(dY)
    N, C = x.shape
    D = C // H
    shared = heads_shared(p)
    dx = np.empty((N, C))
    per = []
    for h in range(H):
        sl = slice(h * D, (h + 1) * D)
        g = layer_backward(x[:, sl], None if G is None else G[h], _head_params(p, h, shared),
                           tau0, tau_min, eps, 1, fwd["heads"][h], dY[:, sl])
        dx[:, sl] = g["dx"]
        per.append(g)
    out = {"dx": dx}
    for k in ("dWq", "dbq", "dWk", "dbk", "dWv", "dbv", "dWo", "dbo", "dtau0"):
        if k in per[0]:
            out[k] = sum(g[k] for g in per)
    for k in ("dA", "db", "da", "db_t"):
        stacked = np.array([g[k] for g in per])
        out[k] = stacked.sum(axis=0) if shared else stacked
    return out

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

from .build import LIB, build

_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build()
        lib = ctypes.CDLL(LIB)
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

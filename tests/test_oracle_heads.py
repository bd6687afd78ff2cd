"""Pins of the per-head slicing oracle (the heads of Eq. 2 carried into the
slicing of Eq. 1: head h slices its own channel block with its own slice
parameters and noise; the token projections are shared by the heads).

Pinned against: the one-head layer (H = 1), the closed form of one slice per
head (the state is the mean of the block and attention over one token returns
its value row), equivariance under a permutation of the heads, and central
finite differences of every gradient, with per-head and shared slice
parameters.
"""
import numpy as np
import pytest

import oracle

RNG = np.random.default_rng(2503)
TAU0, TAU_MIN, EPS = 0.5, 0.01, 1e-5


def _r(*shape, scale=1.0):
    return scale * RNG.standard_normal(shape)


def _params(H, D, M, shared=False, with_o=True, ada=True):
    s = () if shared else (H,)
    p = {"A": _r(*s, D, M, scale=0.4), "b": _r(*s, M, scale=0.2),
         "a": _r(*s, D, scale=0.05) if ada else None,
         "b_t": (0.1 if shared else _r(H, scale=0.05)) if ada else (0.0 if shared else np.zeros(H))}
    for n in ("q", "k", "v") + (("o",) if with_o else ()):
        p["W" + n] = _r(D, D, scale=D ** -0.5)
        p["b" + n] = _r(D, scale=0.1)
    return p


def _gumbel(H, N, M):
    u = RNG.uniform(1e-6, 1.0, size=(H, N, M))
    return -np.log(-np.log(u))


def test_one_head_is_the_layer():
    N, C, M = 300, 16, 8
    x, G = _r(N, C), _gumbel(1, N, M)
    p = _params(1, C, M)
    f = oracle.heads_layer_forward(x, G, p, TAU0, TAU_MIN, EPS, 1)
    q = {k: (v[0] if k in ("A", "b", "a") else v) for k, v in p.items()}
    q["b_t"] = float(p["b_t"][0])
    ref = oracle.layer_forward(x, G[0], q, TAU0, TAU_MIN, EPS, 1)
    np.testing.assert_allclose(f["y"], ref["y"], rtol=0, atol=0)
    dY = _r(N, C)
    g = oracle.heads_layer_backward(x, G, p, TAU0, TAU_MIN, EPS, 1, f, dY)
    gr = oracle.layer_backward(x, G[0], q, TAU0, TAU_MIN, EPS, 1, ref, dY)
    for k in ("dx", "dWq", "dbq", "dWo", "dtau0"):
        np.testing.assert_allclose(g[k], gr[k], rtol=0, atol=0)
    np.testing.assert_allclose(g["dA"][0], gr["dA"], rtol=0, atol=0)
    assert g["db_t"][0] == gr["db_t"]


@pytest.mark.parametrize("with_o", [False, True])
def test_one_slice_per_head_closed_form(with_o):
    """M = 1: every weight is 1, so S_h is the mean of x_h; attention over one
    token returns its value row; every point receives it."""
    N, H, D = 257, 4, 8
    x = _r(N, H * D) + 0.3
    p = _params(H, D, 1, with_o=with_o)
    f = oracle.heads_layer_forward(x, _gumbel(H, N, 1), p, TAU0, TAU_MIN, EPS, H)
    for h in range(H):
        s = x[:, h * D:(h + 1) * D].mean(axis=0)
        v = s @ p["Wv"] + p["bv"]
        if with_o:
            v = v @ p["Wo"] + p["bo"]
        np.testing.assert_allclose(f["y"][:, h * D:(h + 1) * D], np.tile(v, (N, 1)),
                                   rtol=1e-12, atol=1e-13)


def test_heads_permutation_equivariance():
    N, H, D, M = 200, 3, 8, 6
    x, G, p = _r(N, H * D), _gumbel(H, N, M), _params(H, D, M)
    perm = [2, 0, 1]
    cols = np.concatenate([np.arange(h * D, (h + 1) * D) for h in perm])
    q = dict(p)
    for k in ("A", "b", "a", "b_t"):
        q[k] = np.asarray(p[k])[perm]
    f = oracle.heads_layer_forward(x, G, p, TAU0, TAU_MIN, EPS, H)
    fp = oracle.heads_layer_forward(x[:, cols], G[perm], q, TAU0, TAU_MIN, EPS, H)
    np.testing.assert_allclose(fp["y"], f["y"][:, cols], rtol=1e-13, atol=1e-14)
    # a head's output depends on its own block only
    x2 = x.copy()
    x2[:, 0:D] += 1.0
    f2 = oracle.heads_layer_forward(x2, G, p, TAU0, TAU_MIN, EPS, H)
    np.testing.assert_array_equal(f2["y"][:, D:], f["y"][:, D:])
    assert np.abs(f2["y"][:, :D] - f["y"][:, :D]).max() > 1e-3


def _loss(x, G, p, H, dY):
    return float((oracle.heads_layer_forward(x, G, p, TAU0, TAU_MIN, EPS, H)["y"] * dY).sum())


@pytest.mark.parametrize("shared,noise", [(False, True), (True, True), (False, False)])
def test_heads_backward_finite_differences(shared, noise):
    N, H, D, M = 40, 2, 4, 3
    x = _r(N, H * D)
    G = _gumbel(H, N, M) if noise else None
    p = _params(H, D, M, shared=shared, ada=noise)
    dY = _r(N, H * D)
    f = oracle.heads_layer_forward(x, G, p, TAU0, TAU_MIN, EPS, H)
    g = oracle.heads_layer_backward(x, G, p, TAU0, TAU_MIN, EPS, H, f, dY)
    h = 1e-6

    def fd(get, setv, idx):
        base = get()
        plus, minus = base.copy(), base.copy()
        plus[idx] += h
        minus[idx] -= h
        setv(plus)
        lp = _loss(x_cur[0], G, p, H, dY)
        setv(minus)
        lm = _loss(x_cur[0], G, p, H, dY)
        setv(base)
        return (lp - lm) / (2 * h)

    x_cur = [x]
    for idx in [(0, 0), (7, 5), (N - 1, H * D - 1)]:
        got = fd(lambda: x_cur[0], lambda v: x_cur.__setitem__(0, v), idx)
        assert abs(got - g["dx"][idx]) < 1e-6 * max(1.0, abs(got))
    names = ["A", "b", "Wq", "bk", "Wv", "Wo", "bo"] + (["a", "b_t"] if noise else [])
    for k in names:
        arr = np.array(p[k], dtype=np.float64)
        flat = arr.reshape(-1)
        for j in sorted({0, flat.size // 2, flat.size - 1}):
            idx = np.unravel_index(j, arr.shape) if arr.ndim else ()

            def setv(v, k=k):
                p[k] = v if arr.ndim else float(v)
            got = fd(lambda: np.array(p[k], dtype=np.float64), setv, idx)
            want = np.asarray(g["d" + k])[idx] if arr.ndim else float(np.asarray(g["d" + k]))
            assert abs(got - want) < 2e-6 * max(1.0, abs(got)), (k, idx, got, want)
    # the constant temperature's gradient sums over the heads
    got = (_loss_tau(x, G, p, H, dY, TAU0 + h) - _loss_tau(x, G, p, H, dY, TAU0 - h)) / (2 * h)
    assert abs(got - g["dtau0"]) < 2e-6 * max(1.0, abs(got))


def _loss_tau(x, G, p, H, dY, tau0):
    return float((oracle.heads_layer_forward(x, G, p, tau0, TAU_MIN, EPS, H)["y"] * dY).sum())

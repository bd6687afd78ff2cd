"""Pins of the block-stack oracle (LayerNorm, GELU, Linear, the block and the
stack composition) against library routines in float64 (torch), closed
forms and central finite differences; and the Project-folding identity the
GPU path relies on (Algorithm 1's Project step folded into the slice
parameters and the states).
"""
import numpy as np
import pytest
import torch

import oracle

RNG = np.random.default_rng(2502)


def _r(*shape, scale=1.0):
    return scale * RNG.standard_normal(shape)


def _t(a, grad=False):
    return torch.tensor(a, dtype=torch.float64, requires_grad=grad)


# ---------------------------------------------------------------------------
# Pieces against torch's float64 routines
# ---------------------------------------------------------------------------

def test_layernorm_matches_library_and_normalises():
    x, g, b = _r(37, 24, scale=3.0) + 1.5, _r(24), _r(24)
    y, mean, rstd = oracle.layernorm(x, g, b)
    ref = torch.nn.functional.layer_norm(_t(x), (24,), _t(g), _t(b), eps=oracle.LN_EPS)
    np.testing.assert_allclose(y, ref.numpy(), rtol=0, atol=1e-12)
    y1, _, _ = oracle.layernorm(x, None, None)
    np.testing.assert_allclose(y1.mean(axis=1), 0.0, atol=1e-13)
    var = x.var(axis=1)
    np.testing.assert_allclose((y1 ** 2).mean(axis=1), var / (var + oracle.LN_EPS), rtol=1e-12)
    np.testing.assert_allclose(mean, x.mean(axis=1), rtol=1e-13)
    np.testing.assert_allclose(rstd, 1.0 / np.sqrt(var + oracle.LN_EPS), rtol=1e-12)


def test_layernorm_backward_matches_autograd():
    x, g, b, dy = _r(1500, 16), _r(16), _r(16), _r(1500, 16)   # > one shard of points
    xt, gt, bt = _t(x, True), _t(g, True), _t(b, True)
    torch.nn.functional.layer_norm(xt, (16,), gt, bt, eps=oracle.LN_EPS).backward(_t(dy))
    dx, dg, db = oracle.layernorm_backward(x, g, dy)
    np.testing.assert_allclose(dx, xt.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dg, gt.grad.numpy(), rtol=1e-10)
    np.testing.assert_allclose(db, bt.grad.numpy(), rtol=1e-10)


def test_gelu():
    x = np.concatenate([_r(500, scale=3.0), [0.0, 8.0, -8.0, 1.0]])
    y = oracle.gelu(x)
    # the standard normal CDF at 1 (a tabulated value): GELU(1) = Phi(1)
    assert abs(y[-1] - 0.8413447460685429) < 1e-15
    assert y[-4] == 0.0 and abs(y[-3] - 8.0) < 1e-13 and abs(y[-2]) < 1e-13
    # Phi(x) + Phi(-x) = 1, so GELU(x) - GELU(-x) = x
    np.testing.assert_allclose(y[:500] - oracle.gelu(-x[:500]), x[:500], rtol=1e-14,
                               atol=1e-14)
    ref = torch.nn.functional.gelu(_t(x), approximate="none").numpy()
    np.testing.assert_allclose(y, ref, rtol=1e-14, atol=1e-16)
    # GELU'(0) = 1/2; derivative against autograd and central differences
    dy = _r(x.size)
    xt = _t(x, True)
    torch.nn.functional.gelu(xt, approximate="none").backward(_t(dy))
    np.testing.assert_allclose(oracle.gelu_backward(x, dy), xt.grad.numpy(), rtol=1e-12,
                               atol=1e-14)
    assert oracle.gelu_backward(np.array([0.0]), np.array([1.0]))[0] == 0.5
    h = 1e-6
    fd = (oracle.gelu(x[:50] + h) - oracle.gelu(x[:50] - h)) / (2 * h)
    np.testing.assert_allclose(oracle.gelu_backward(x[:50], np.ones(50)), fd, rtol=1e-8,
                               atol=1e-9)


def test_linear_and_backward():
    # brute force on a tiny case: every output an explicit sum
    xs, Ws, bs = _r(3, 4), _r(4, 5), _r(5)
    brute = np.array([[bs[o] + sum(xs[i, k] * Ws[k, o] for k in range(4)) for o in range(5)]
                      for i in range(3)])
    np.testing.assert_allclose(oracle.linear(xs, Ws, bs), brute, rtol=1e-14, atol=1e-14)
    x, W, b, dy = _r(1300, 12), _r(12, 20), _r(20), _r(1300, 20)
    np.testing.assert_allclose(oracle.linear(x, W, b),
                               torch.nn.functional.linear(_t(x), _t(W).T, _t(b)).numpy(),
                               rtol=1e-12, atol=1e-12)
    xt, Wt, bt = _t(x, True), _t(W, True), _t(b, True)
    (xt @ Wt + bt).backward(_t(dy))
    dx, dW, db = oracle.linear_backward(x, W, dy)
    np.testing.assert_allclose(dx, xt.grad.numpy(), rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(dW, Wt.grad.numpy(), rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(db, bt.grad.numpy(), rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------------------
# Block and stack: central finite differences of the composition
# ---------------------------------------------------------------------------

def block_params(C, M, rng, scale=0.4):
    r = lambda *s, sc=scale: sc * rng.standard_normal(s)
    return {
        "A": r(C, M, sc=0.7), "b": r(M, sc=0.3), "a": r(C, sc=0.05), "b_t": 0.05,
        "Wq": r(C, C), "bq": r(C, sc=0.1), "Wk": r(C, C), "bk": r(C, sc=0.1),
        "Wv": r(C, C), "bv": r(C, sc=0.1), "Wo": r(C, C), "bo": r(C, sc=0.1),
        "ln1_g": 1.0 + r(C, sc=0.1), "ln1_b": r(C, sc=0.1), "Wp": r(C, C), "bp": r(C, sc=0.1),
        "ln2_g": 1.0 + r(C, sc=0.1), "ln2_b": r(C, sc=0.1),
        "W1": r(C, 4 * C), "b1": r(4 * C, sc=0.1), "W2": r(4 * C, C, sc=0.2), "b2": r(C, sc=0.1),
    }


SHAPE = dict(N=24, C=8, M=3, H=2)
TAU0, TAU_MIN, EPS = 0.5, 0.01, 1e-5


def _fd(f, theta, v, h=1e-6):
    return (f(theta + h * v) - f(theta - h * v)) / (2 * h)


@pytest.mark.parametrize("name", ["x", "W1", "Wp", "ln1_g", "A", "a", "Wq", "Wo", "b2"])
def test_block_backward_finite_differences(name):
    rng = np.random.default_rng(7)
    N, C, M, H = SHAPE["N"], SHAPE["C"], SHAPE["M"], SHAPE["H"]
    p = block_params(C, M, rng)
    x = rng.standard_normal((N, C))
    G = -np.log(-np.log(rng.uniform(1e-6, 1.0, (N, M))))
    dy = rng.standard_normal((N, C))
    out, cache = oracle.block_forward(x, G, p, TAU0, TAU_MIN, EPS, H)
    assert np.all(cache["pa"]["tau"] > TAU_MIN)  # away from the clamp
    dx, grads = oracle.block_backward(dy, G, p, TAU0, TAU_MIN, EPS, H, cache)

    base = x if name == "x" else p[name]
    v = rng.standard_normal(np.shape(base))

    def loss(theta):
        if name == "x":
            o, _ = oracle.block_forward(theta, G, p, TAU0, TAU_MIN, EPS, H)
        else:
            q = dict(p)
            q[name] = theta
            o, _ = oracle.block_forward(x, G, q, TAU0, TAU_MIN, EPS, H)
        return float(np.sum(o * dy))

    fd = _fd(loss, np.asarray(base, dtype=np.float64), v)
    g = dx if name == "x" else grads["d" + name]
    an = float(np.sum(g * v))
    assert abs(an - fd) <= 1e-6 * max(1.0, abs(fd)), (name, an, fd)


def test_stack_backward_finite_differences():
    rng = np.random.default_rng(11)
    N, C, M, H = SHAPE["N"], SHAPE["C"], SHAPE["M"], SHAPE["H"]
    ps = [block_params(C, M, rng) for _ in range(2)]
    Gs = [-np.log(-np.log(rng.uniform(1e-6, 1.0, (N, M)))) for _ in range(2)]
    x = rng.standard_normal((N, C))
    dy = rng.standard_normal((N, C))
    out, caches = oracle.stack_forward(x, Gs, ps, TAU0, TAU_MIN, EPS, H)
    dx, grads = oracle.stack_backward(dy, Gs, ps, TAU0, TAU_MIN, EPS, H, caches)
    assert len(grads) == 2 and set(grads[0]) == set(grads[1])
    v = rng.standard_normal(x.shape)
    f = lambda t: float(np.sum(oracle.stack_forward(t, Gs, ps, TAU0, TAU_MIN, EPS, H)[0] * dy))
    fd = _fd(f, x, v)
    assert abs(float(np.sum(dx * v)) - fd) <= 1e-6 * max(1.0, abs(fd))
    # the second block's input is the first block's output
    o1, _ = oracle.block_forward(x, Gs[0], ps[0], TAU0, TAU_MIN, EPS, H)
    o2, _ = oracle.block_forward(o1, Gs[1], ps[1], TAU0, TAU_MIN, EPS, H)
    np.testing.assert_array_equal(out, o2)


def test_block_reduces_to_its_parts():
    """With W1 = 0 (MLP = b2) the block is x + PA(LN1(x) Wp + bp) + b2."""
    rng = np.random.default_rng(3)
    N, C, M, H = 40, 8, 4, 2
    p = block_params(C, M, rng)
    p["W1"] = np.zeros_like(p["W1"])
    x = rng.standard_normal((N, C))
    G = -np.log(-np.log(rng.uniform(1e-6, 1.0, (N, M))))
    out, _ = oracle.block_forward(x, G, p, TAU0, TAU_MIN, EPS, H)
    h, _, _ = oracle.layernorm(x, p["ln1_g"], p["ln1_b"])
    y = oracle.layer_forward(h @ p["Wp"] + p["bp"], G, p, TAU0, TAU_MIN, EPS, H)["y"]
    g0 = oracle.gelu(p["b1"])                  # GELU(0 + b1) for every row
    np.testing.assert_allclose(out, x + y + g0 @ p["W2"] + p["b2"], rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------------------
# The folding identity of the GPU path (Algorithm 1's Project step)
# ---------------------------------------------------------------------------

def test_project_folds_into_slice_parameters_and_states():
    """x_proj = h Wp + bp.  The logits and temperature of x_proj equal those
    of h under A' = Wp A, b' = b + bp A, a' = Wp a, b_t' = b_t + bp.a; the
    states of x_proj equal S(h) Wp + bp wherever den >= eps (the weights of
    a point sum to 1); so the layer on x_proj is the folded layer on h."""
    rng = np.random.default_rng(5)
    N, C, M, H = 300, 16, 5, 4
    p = block_params(C, M, rng)
    h = rng.standard_normal((N, C))
    G = -np.log(-np.log(rng.uniform(1e-6, 1.0, (N, M))))
    xp = h @ p["Wp"] + p["bp"]
    ref = oracle.layer_forward(xp, G, p, TAU0, TAU_MIN, EPS, H)
    Af, bf = p["Wp"] @ p["A"], p["b"] + p["bp"] @ p["A"]
    af, btf = p["Wp"] @ p["a"], p["b_t"] + float(p["bp"] @ p["a"])
    W, _, _ = oracle.slice_weights(h, G, Af, bf, af, btf, TAU0, TAU_MIN)
    np.testing.assert_allclose(W, ref["W"], rtol=1e-11, atol=1e-13)
    _, den, S = oracle.aggregate(h, W, EPS)
    assert np.all(den >= EPS)
    Sproj = S @ p["Wp"] + p["bp"]
    np.testing.assert_allclose(Sproj, ref["S"], rtol=1e-11, atol=1e-12)
    Sp = oracle.token_attention(Sproj, H, p["Wq"], p["bq"], p["Wk"], p["bk"], p["Wv"], p["bv"],
                                p["Wo"], p["bo"])
    np.testing.assert_allclose(oracle.deslice(W, Sp), ref["y"], rtol=1e-10, atol=1e-12)

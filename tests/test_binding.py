"""The Python binding's argument checks and marshalling, on the CPU.

The library itself is replaced by a recorder (no pointer is dereferenced and
nothing is launched), and host tensors stand in for device tensors: every
wrapper of a layer call must accept tensors of exactly the sizes its dims
describe, pass one argument per parameter of the C declaration, and refuse
a tensor that is too small or of the wrong dtype before calling the library.
"""
import ctypes

import pytest
import torch

from paper_2502_02414_amd import binding as B


class _Recorder:
    def __init__(self):
        self.calls = []

    def __getattr__(self, name):
        def call(*args):
            self.calls.append((name, args))
            return B.PA_OK
        return call

    def pa_last_error(self):
        return b""


@pytest.fixture
def fake(monkeypatch):
    rec = _Recorder()
    monkeypatch.setattr(B, "load", lambda *a, **k: rec)
    monkeypatch.setattr(B, "_ptr", lambda t: None if t is None else 4096)
    monkeypatch.setattr(B, "_stream", lambda s=None: None)
    return rec


N, C, H, M = 100, 32, 2, 8


def _t(*shape, dt=torch.float32):
    return torch.zeros(*shape, dtype=dt)


@pytest.mark.parametrize("dt", [B.PA_F32, B.PA_BF16])
def test_layer_calls_accept_their_shapes(fake, dt):
    tdt = torch.bfloat16 if dt == B.PA_BF16 else torch.float32
    d = B.make_dims(N, C, H, M, 0.5, 0.01, 1e-5, dt)
    x, G, y = _t(N, C, dt=tdt), _t(N, M, dt=tdt), _t(N, C, dt=tdt)
    sp = B.make_slice_params(_t(C, M, dt=tdt), _t(M), _t(C, dt=tdt), 0.1, _t(1))
    ap = B.make_attn_params(_t(C, C), _t(C, C), _t(C, C), _t(C), _t(C), _t(C), _t(C, C), _t(C))
    mc, m = _t(M, C), _t(M)
    ws = _t(64, dt=torch.uint8)
    gr = B.make_slice_grads(_t(C, M), _t(M), _t(C), _t(1), _t(1))
    ag = B.make_attn_grads(*[_t(C, C) if i % 2 == 0 else _t(C) for i in range(8)])
    B.pa_slice_weights(d, x, G, sp, _t(N, M), _t(N), ws)
    B.pa_slice_aggregate(d, x, G, sp, mc, m, mc, ws)
    B.pa_token_attention(d, mc, ap, mc, ws)
    B.pa_deslice(d, x, G, sp, mc, y, ws)
    B.pa_deslice_backward(d, x, G, sp, y, mc, ws)
    B.pa_token_attention_backward(d, mc, ap, mc, mc, ag, ws)
    B.pa_slice_aggregate_backward(d, x, G, sp, mc, m, mc, mc, y, y, gr, ws)
    B.pa_slice_weights_backward(d, x, G, sp, _t(N, M), _t(N), y, gr, ws)
    B.pa_slice_aggregate_w(d, x, G, sp, mc, m, mc, _t(N, M, dt=tdt), ws)
    B.pa_deslice_w(d, _t(N, M, dt=tdt), mc, y, ws)
    B.pa_deslice_backward_w(d, _t(N, M, dt=tdt), y, mc, ws)
    B.pa_slice_aggregate_noalloc(d, x, G, sp, mc, m, mc)
    # one argument per parameter of each C declaration
    nargs = {name: len(args) for name, args in fake.calls}
    assert nargs == {"pa_slice_weights": 9, "pa_slice_aggregate": 10, "pa_token_attention": 7,
                     "pa_deslice": 9, "pa_deslice_backward": 9,
                     "pa_token_attention_backward": 9, "pa_slice_aggregate_backward": 14,
                     "pa_slice_weights_backward": 11, "pa_slice_aggregate_w": 11,
                     "pa_deslice_w": 7, "pa_deslice_backward_w": 7,
                     "pa_slice_aggregate_noalloc": 8}


def test_heads_calls_accept_their_shapes(fake):
    heads, D = 4, 32
    d = B.make_dims(N, D, 1, M, 0.5, 0.01, 1e-5, B.PA_F32)
    x, G = _t(heads, N, D), _t(heads, N, M)
    hp = B.make_heads_params(_t(heads, D, M), _t(heads, M), _t(heads, D), _t(heads))
    mc, m, ws = _t(heads, M, D), _t(heads, M), _t(64, dt=torch.uint8)
    gr = B.make_slice_grads(_t(heads, D, M), _t(heads, M), _t(heads, D), _t(heads), _t(heads))
    B.pa_heads_slice_aggregate(d, heads, x, G, hp, mc, m, mc, ws)
    B.pa_heads_deslice(d, heads, x, G, hp, mc, x, ws)
    B.pa_heads_deslice_backward(d, heads, x, G, hp, x, mc, ws)
    B.pa_heads_slice_aggregate_backward(d, heads, x, G, hp, mc, m, mc, mc, x, x, gr, ws)
    shared = B.make_heads_params(_t(D, M), _t(M), _t(D), _t(1), shared=True)
    B.pa_heads_slice_aggregate(d, heads, x, G, shared, mc, m, mc, ws)
    # a per-head parameter block too small for the heads
    small = B.make_heads_params(_t(heads - 1, D, M))
    with pytest.raises(ValueError, match="A"):
        B.pa_heads_slice_aggregate(d, heads, x, G, small, mc, m, mc, ws)
    with pytest.raises(ValueError, match="x"):
        B.pa_heads_deslice(d, heads, x[:2], G, hp, mc, x, ws)
    # per-head gradients are stacked head after head
    gr1 = B.make_slice_grads(_t(D, M))
    with pytest.raises(ValueError, match="dA"):
        B.pa_heads_slice_aggregate_backward(d, heads, x, G, hp, mc, m, mc, mc, x, x, gr1, ws)


def test_small_or_mistyped_tensors_refused_before_the_call(fake):
    d = B.make_dims(N, C, H, M, 0.5, 0.01, 1e-5, B.PA_BF16)
    bf = torch.bfloat16
    x, G, ws = _t(N, C, dt=bf), _t(N, M, dt=bf), _t(64, dt=torch.uint8)
    sp = B.make_slice_params(_t(C, M, dt=bf))
    mc, m = _t(M, C), _t(M)
    with pytest.raises(ValueError, match="x"):
        B.pa_slice_aggregate(d, x[:-1], G, sp, mc, m, mc, ws)
    with pytest.raises(ValueError, match="dtype"):
        B.pa_slice_aggregate(d, x.float(), G, sp, mc, m, mc, ws)
    with pytest.raises(ValueError, match="den"):
        B.pa_slice_aggregate(d, x, G, sp, mc, m[:-1], mc, ws)
    with pytest.raises(ValueError, match="A"):
        B.pa_slice_aggregate(d, x, G, B.make_slice_params(_t(C, M)), mc, m, mc, ws)
    with pytest.raises(ValueError, match="Wq"):
        B.pa_token_attention(d, mc, B.make_attn_params(_t(C, C - 1), _t(C, C), _t(C, C)), mc, ws)
    with pytest.raises(ValueError, match="dA"):
        B.pa_slice_aggregate_backward(d, x, G, sp, mc, m, mc, None, None, x,
                                      B.make_slice_grads(dA=_t(C * M - 1)), ws)
    assert fake.calls == []


def test_wrapper_calls_match_argtypes():
    """Every load().pa_*(...) call in the binding passes exactly as many
    arguments as the symbol's ctypes argtypes declare (read from the source,
    no GPU needed)."""
    import ast
    import inspect
    from paper_2502_02414_amd import binding as B
    lib = B.load()
    tree = ast.parse(inspect.getsource(B))
    calls = 0
    for node in ast.walk(tree):
        if not (isinstance(node, ast.Call) and isinstance(node.func, ast.Attribute)):
            continue
        f = node.func
        if isinstance(f.value, ast.Call) and getattr(f.value.func, "id", "") == "load" \
                and f.attr.startswith("pa_"):
            calls += 1
            assert len(node.args) == len(getattr(lib, f.attr).argtypes or []), f.attr
    assert calls > 30
    # pa_gemm and pa_gemm_prepare are called through a chosen function
    assert lib.pa_gemm.argtypes == lib.pa_gemm_prepare.argtypes
    src = inspect.getsource(B.pa_gemm)
    call = next(n for n in ast.walk(ast.parse(src.strip()))
                if isinstance(n, ast.Call) and getattr(n.func, "id", "") == "fn")
    assert len(call.args) == len(lib.pa_gemm.argtypes)

"""Thin Python binding of the C ABI in include/pa.h (``libpa.so``).

Same entry-point names as the C library; each wrapper only checks and
marshals arguments (torch device tensors -> device pointers, the current
HIP stream) and raises ``PAError`` on a non-zero status.  Every step of the
layer runs in the library's HIP kernels; there is no fallback of any kind:
if ``libpa.so`` is missing or no GPU is present, calls fail loudly.

Tensors: row-major contiguous CUDA (HIP) tensors.  Point-side tensors
(x, G, y, dY, dx) and the slice projection (A, a) are ``torch.float32`` or
``torch.bfloat16`` (matching ``dims.dtype``); tokens, b, attention
parameters and every gradient of a parameter are float32.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libpa.so")

PA_F32, PA_BF16 = 0, 1
PA_OK, PA_ERR_INVALID, PA_ERR_UNSUPPORTED, PA_ERR_WORKSPACE, PA_ERR_HIP = 0, -1, -2, -3, -4

# every exported symbol declared in include/pa.h
SYMBOLS = (
    "pa_version", "pa_last_error", "pa_workspace_size", "pa_slice_weights",
    "pa_slice_aggregate", "pa_token_attention", "pa_deslice", "pa_deslice_backward",
    "pa_token_attention_backward", "pa_slice_aggregate_backward",
    "pa_slice_weights_backward", "pa_time_kernel", "pa_slice_aggregate_w", "pa_deslice_w",
    "pa_deslice_backward_w", "pa_gemm", "pa_layernorm", "pa_layernorm_backward", "pa_gelu",
    "pa_gelu_backward", "pa_colsum", "pa_project_fold", "pa_project_states",
    "pa_project_backward", "pa_heads_relayout", "pa_heads_expand", "pa_heads_sum",
    "pa_heads_workspace_size", "pa_heads_slice_aggregate", "pa_heads_deslice",
    "pa_heads_deslice_backward", "pa_heads_slice_aggregate_backward",
    "pa_slice_aggregate_noalloc", "pa_mlp_up", "pa_mlp_up_backward", "pa_gemm_prepare",
    "pa_stream_probe", "pa_heads_sum_batch",
)


class PAError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"pa status {status}: {msg}")
        self.status = status


class pa_dims(ctypes.Structure):
    _fields_ = [("N", ctypes.c_int64), ("C", ctypes.c_int32), ("H", ctypes.c_int32),
                ("M", ctypes.c_int32), ("tau0", ctypes.c_float), ("tau_min", ctypes.c_float),
                ("eps", ctypes.c_float), ("dtype", ctypes.c_int32)]


class pa_slice_params(ctypes.Structure):
    _fields_ = [("A", ctypes.c_void_p), ("b", ctypes.c_void_p), ("a", ctypes.c_void_p),
                ("b_t", ctypes.c_float), ("b_t_dev", ctypes.c_void_p)]


class pa_attn_params(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("Wq", "bq", "Wk", "bk", "Wv", "bv", "Wo", "bo")]


class pa_slice_grads(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("dA", "db", "da", "db_t", "dtau0")]


class pa_heads_params(ctypes.Structure):
    _fields_ = [("A", ctypes.c_void_p), ("b", ctypes.c_void_p), ("a", ctypes.c_void_p),
                ("b_t", ctypes.c_void_p), ("shared", ctypes.c_int)]


class pa_attn_grads(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p)
                for n in ("dWq", "dbq", "dWk", "dbk", "dWv", "dbv", "dWo", "dbo")]


class pa_heads_sum_item(ctypes.Structure):
    _fields_ = [("src", ctypes.c_void_p), ("dst", ctypes.c_void_p), ("L", ctypes.c_int64),
                ("blockdiag", ctypes.c_int)]


_lib = None


def load(path: str = LIB_PATH):
    """Load libpa.so (built by ``paper_2502_02414_amd.build``); raises if absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"HIP library {path} is not built; run __graft_entry__.build()")
    # torch's HIP runtime and hipBLASLt are loaded first, so libpa.so binds to
    # the same copies (one HIP runtime per process)
    import torch  # noqa: F401
    lib = ctypes.CDLL(path)
    P, S = ctypes.c_void_p, ctypes.c_size_t
    D = ctypes.POINTER(pa_dims)
    lib.pa_version.restype = ctypes.c_int
    lib.pa_last_error.restype = ctypes.c_char_p
    lib.pa_workspace_size.argtypes = [D, ctypes.POINTER(ctypes.c_size_t)]
    SPp = ctypes.POINTER(pa_slice_params)
    APp = ctypes.POINTER(pa_attn_params)
    SGp = ctypes.POINTER(pa_slice_grads)
    AGp = ctypes.POINTER(pa_attn_grads)
    lib.pa_slice_weights.argtypes = [D, P, P, SPp, P, P, P, S, P]
    lib.pa_slice_aggregate.argtypes = [D, P, P, SPp, P, P, P, P, S, P]
    lib.pa_token_attention.argtypes = [D, P, APp, P, P, S, P]
    lib.pa_deslice.argtypes = [D, P, P, SPp, P, P, P, S, P]
    lib.pa_deslice_backward.argtypes = [D, P, P, SPp, P, P, P, S, P]
    lib.pa_token_attention_backward.argtypes = [D, P, APp, P, P, AGp, P, S, P]
    lib.pa_slice_aggregate_backward.argtypes = [D, P, P, SPp, P, P, P, P, P, P, SGp, P, S, P]
    lib.pa_slice_weights_backward.argtypes = [D, P, P, SPp, P, P, P, SGp, P, S, P]
    lib.pa_time_kernel.argtypes = [ctypes.c_char_p, P, P]
    lib.pa_stream_probe.argtypes = [D, ctypes.c_char_p, P, P, P, P, P]
    lib.pa_slice_aggregate_w.argtypes = [D, P, P, SPp, P, P, P, P, P, S, P]
    lib.pa_slice_aggregate_noalloc.argtypes = [D, P, P, SPp, P, P, P, P]
    lib.pa_deslice_w.argtypes = [D, P, P, P, P, S, P]
    lib.pa_deslice_backward_w.argtypes = [D, P, P, P, P, S, P]
    I64, I32, F = ctypes.c_int64, ctypes.c_int, ctypes.c_float
    lib.pa_gemm.argtypes = [I32, I32, I64, I64, I64, F, P, I32, P, I32, F, P, P, I32, P, P, S, P]
    lib.pa_gemm_prepare.argtypes = lib.pa_gemm.argtypes
    lib.pa_layernorm.argtypes = [I64, I32, F, I32, P, P, P, P, P, P, P, P, P]
    lib.pa_layernorm_backward.argtypes = [I64, I32, I32, P, P, P, P, P, P, P, P, P, P, S, P]
    lib.pa_gelu.argtypes = [I64, I32, P, P, P]
    lib.pa_gelu_backward.argtypes = [I64, I32, P, P, P, P]
    lib.pa_colsum.argtypes = [I64, I32, I32, P, P, P, S, P]
    lib.pa_mlp_up.argtypes = [I64, I32, I32, P, P, P, P, P, S, P]
    lib.pa_mlp_up_backward.argtypes = [I64, I32, I32, P, P, P, P, P, P, P, S, P]
    lib.pa_project_fold.argtypes = [D, P, P, P, P, P, P, P, P, P, P]
    lib.pa_project_states.argtypes = [D, P, P, P, P, P]
    lib.pa_project_backward.argtypes = [D, P, P, P, P, P, P, SGp, P, P, P, SGp, P]
    lib.pa_heads_relayout.argtypes = [I64, I32, I32, I32, I32, P, P, P]
    lib.pa_heads_expand.argtypes = [I32, I64, I32, P, P, P]
    lib.pa_heads_sum.argtypes = [I32, I64, I32, P, P, P]
    lib.pa_heads_sum_batch.argtypes = [I32, I32, ctypes.POINTER(pa_heads_sum_item), P]
    HPp = ctypes.POINTER(pa_heads_params)
    lib.pa_heads_workspace_size.argtypes = [D, I32, ctypes.POINTER(ctypes.c_size_t)]
    lib.pa_heads_slice_aggregate.argtypes = [D, I32, P, P, HPp, P, P, P, P, S, P]
    lib.pa_heads_deslice.argtypes = [D, I32, P, P, HPp, P, P, P, S, P]
    lib.pa_heads_deslice_backward.argtypes = [D, I32, P, P, HPp, P, P, P, S, P]
    lib.pa_heads_slice_aggregate_backward.argtypes = [D, I32, P, P, HPp, P, P, P, P, P, P, SGp,
                                                      P, S, P]
    for name in SYMBOLS:
        if name not in ("pa_version", "pa_last_error"):
            getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def _check(status: int):
    if status != PA_OK:
        raise PAError(status, load().pa_last_error().decode())


def _ptr(t) -> Optional[int]:
    """Device pointer of a contiguous CUDA tensor (or None)."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("tensor must be on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    return t.data_ptr()


# Element-count and dtype checks against the dims of a call: the library
# only sees pointers, so a tensor smaller than the shape it stands for would
# be read or written past its end.  A requirement is (elements, dtype), the
# dtype a PA_* code, or None for "fp32 or the storage dtype" (not checked).
def _need(t, n: int, dt: Optional[int], name: str):
    if t is None:
        return
    if t.numel() < n:
        raise ValueError(f"{name}: {t.numel()} elements, the call needs {n}")
    if dt is not None and _dt(t) != dt:
        raise ValueError(f"{name}: dtype {t.dtype} does not match the call's "
                         f"{'bf16' if dt == PA_BF16 else 'fp32'}")


def _arg(t, n: int, dt: Optional[int], name: str) -> Optional[int]:
    """Pointer of t after checking it against (n elements, dtype dt)."""
    _need(t, n, dt, name)
    return _ptr(t)


def _check_struct(st, dims, heads: int = 1, stacked: bool = False):
    """Checks the tensors a parameter struct was made from against dims
    (structs built by the make_* helpers below carry their tensors);
    ``stacked``: every tensor holds one block per head."""
    for name, (t, kind) in getattr(st, "_tensors", {}).items():
        n = _struct_count(kind, dims, heads) * (heads if stacked else 1)
        _need(t, n, _struct_dtype(kind, dims), name)


def _struct_count(kind: str, d, heads: int) -> int:
    C, M = d.C, d.M
    return {"CM": C * M, "CM32": C * M, "M": M, "C": C, "C32": C, "1": 1, "CC": C * C,
            "hCM": heads * C * M, "hCM32": heads * C * M, "hM": heads * M, "hC": heads * C,
            "hC32": heads * C, "h": heads}[kind]


def _struct_dtype(kind: str, d) -> Optional[int]:
    # A and a are in the storage dtype; everything else in the structs is fp32
    return {"CM": d.dtype, "C": d.dtype, "hCM": d.dtype, "hC": d.dtype}.get(kind, PA_F32)


def _with(st, **tensors):
    st._tensors = {k: v for k, v in tensors.items() if v[0] is not None}
    return st


def _stream(stream=None) -> Optional[int]:
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def make_dims(N: int, C: int, H: int, M: int, tau0: float, tau_min: float, eps: float,
              dtype: int) -> pa_dims:
    return pa_dims(int(N), int(C), int(H), int(M), float(tau0), float(tau_min), float(eps),
                   int(dtype))


def make_slice_params(A, b=None, a=None, b_t: float = 0.0, b_t_dev=None) -> pa_slice_params:
    return _with(pa_slice_params(_ptr(A), _ptr(b), _ptr(a), float(b_t), _ptr(b_t_dev)),
                 A=(A, "CM"), b=(b, "M"), a=(a, "C"), b_t_dev=(b_t_dev, "1"))


def make_attn_params(Wq, Wk, Wv, bq=None, bk=None, bv=None, Wo=None, bo=None) -> pa_attn_params:
    return _with(pa_attn_params(_ptr(Wq), _ptr(bq), _ptr(Wk), _ptr(bk), _ptr(Wv), _ptr(bv),
                                _ptr(Wo), _ptr(bo)),
                 Wq=(Wq, "CC"), Wk=(Wk, "CC"), Wv=(Wv, "CC"), Wo=(Wo, "CC"), bq=(bq, "C32"),
                 bk=(bk, "C32"), bv=(bv, "C32"), bo=(bo, "C32"))


def make_slice_grads(dA=None, db=None, da=None, db_t=None, dtau0=None) -> pa_slice_grads:
    return _with(pa_slice_grads(_ptr(dA), _ptr(db), _ptr(da), _ptr(db_t), _ptr(dtau0)),
                 dA=(dA, "CM32"), db=(db, "M"), da=(da, "C32"), db_t=(db_t, "1"),
                 dtau0=(dtau0, "1"))


def make_attn_grads(dWq=None, dbq=None, dWk=None, dbk=None, dWv=None, dbv=None, dWo=None,
                    dbo=None) -> pa_attn_grads:
    return _with(pa_attn_grads(_ptr(dWq), _ptr(dbq), _ptr(dWk), _ptr(dbk), _ptr(dWv), _ptr(dbv),
                               _ptr(dWo), _ptr(dbo)),
                 dWq=(dWq, "CC"), dWk=(dWk, "CC"), dWv=(dWv, "CC"), dWo=(dWo, "CC"),
                 dbq=(dbq, "C32"), dbk=(dbk, "C32"), dbv=(dbv, "C32"), dbo=(dbo, "C32"))


def _shapes(dims, heads: int = 1) -> dict:
    """(elements, dtype) of the tensors of a layer call at these dims; with
    heads > 1 the point-side tensors and the states are stacked per head."""
    N, C, M, dt = int(dims.N), int(dims.C), int(dims.M), int(dims.dtype)
    h = int(heads)
    return {"x": (h * N * C, dt), "G": (h * N * M, dt), "W32": (N * M, PA_F32),
            "N32": (N, PA_F32), "MC": (h * M * C, PA_F32), "M": (h * M, PA_F32)}


def pa_version() -> int:
    return load().pa_version()


def pa_last_error() -> str:
    return load().pa_last_error().decode()


def pa_workspace_size(dims: pa_dims) -> int:
    n = ctypes.c_size_t(0)
    _check(load().pa_workspace_size(ctypes.byref(dims), ctypes.byref(n)))
    return n.value


def workspace(dims: pa_dims, device="cuda"):
    """A uint8 device tensor of pa_workspace_size bytes (torch allocates)."""
    import torch
    return torch.empty(pa_workspace_size(dims), dtype=torch.uint8, device=device)


def pa_slice_weights(dims, x, G, sp, W, tau, ws, stream=None):
    d = _shapes(dims)
    _check_struct(sp, dims)
    _check(load().pa_slice_weights(ctypes.byref(dims), _arg(x, *d["x"], "x"), _arg(G, *d["G"], "G"),
                                   ctypes.byref(sp), _arg(W, *d["W32"], "W"), _arg(tau, *d["N32"], "tau"),
                                   _ptr(ws), ws.numel(), _stream(stream)))


def pa_slice_aggregate(dims, x, G, sp, num, den, S, ws, stream=None):
    d = _shapes(dims)
    _check_struct(sp, dims)
    _check(load().pa_slice_aggregate(ctypes.byref(dims), _arg(x, *d["x"], "x"), _arg(G, *d["G"], "G"),
                                     ctypes.byref(sp), _arg(num, *d["MC"], "num"), _arg(den, *d["M"], "den"),
                                     _arg(S, *d["MC"], "S"), _ptr(ws), ws.numel(), _stream(stream)))


def pa_token_attention(dims, S, ap, Sp, ws, stream=None):
    d = _shapes(dims)
    _check_struct(ap, dims)
    _check(load().pa_token_attention(ctypes.byref(dims), _arg(S, *d["MC"], "S"), ctypes.byref(ap),
                                     _arg(Sp, *d["MC"], "Sp"), _ptr(ws), ws.numel(), _stream(stream)))


def pa_deslice(dims, x, G, sp, Sp, y, ws, stream=None):
    d = _shapes(dims)
    _check_struct(sp, dims)
    _check(load().pa_deslice(ctypes.byref(dims), _arg(x, *d["x"], "x"), _arg(G, *d["G"], "G"),
                             ctypes.byref(sp), _arg(Sp, *d["MC"], "Sp"), _arg(y, *d["x"], "y"), _ptr(ws),
                             ws.numel(), _stream(stream)))


def pa_deslice_backward(dims, x, G, sp, dY, dSp, ws, stream=None):
    d = _shapes(dims)
    _check_struct(sp, dims)
    _check(load().pa_deslice_backward(ctypes.byref(dims), _arg(x, *d["x"], "x"), _arg(G, *d["G"], "G"),
                                      ctypes.byref(sp), _arg(dY, *d["x"], "dY"), _arg(dSp, *d["MC"], "dSp"),
                                      _ptr(ws), ws.numel(), _stream(stream)))


def pa_token_attention_backward(dims, S, ap, dSp, dS, ag, ws, stream=None):
    d = _shapes(dims)
    _check_struct(ap, dims)
    if ag is not None:
        _check_struct(ag, dims)
    _check(load().pa_token_attention_backward(
        ctypes.byref(dims), _arg(S, *d["MC"], "S"), ctypes.byref(ap), _arg(dSp, *d["MC"], "dSp"),
        _arg(dS, *d["MC"], "dS"),
        ctypes.byref(ag) if ag is not None else None, _ptr(ws), ws.numel(), _stream(stream)))


def pa_slice_aggregate_backward(dims, x, G, sp, num, den, dS, Sp, dY, dx, gr, ws, stream=None):
    d = _shapes(dims)
    _check_struct(sp, dims)
    if gr is not None:
        _check_struct(gr, dims)
    _check(load().pa_slice_aggregate_backward(
        ctypes.byref(dims), _arg(x, *d["x"], "x"), _arg(G, *d["G"], "G"), ctypes.byref(sp),
        _arg(num, *d["MC"], "num"), _arg(den, *d["M"], "den"), _arg(dS, *d["MC"], "dS"), _arg(Sp, *d["MC"], "Sp"),
        _arg(dY, *d["x"], "dY"), _arg(dx, *d["x"], "dx"), ctypes.byref(gr) if gr is not None else None,
        _ptr(ws), ws.numel(), _stream(stream)))


def pa_slice_weights_backward(dims, x, G, sp, dW, dtau, dx, gr, ws, stream=None):
    d = _shapes(dims)
    _check_struct(sp, dims)
    if gr is not None:
        _check_struct(gr, dims)
    _check(load().pa_slice_weights_backward(
        ctypes.byref(dims), _arg(x, *d["x"], "x"), _arg(G, *d["G"], "G"), ctypes.byref(sp),
        _arg(dW, *d["W32"], "dW"), _arg(dtau, *d["N32"], "dtau"), _arg(dx, *d["x"], "dx"),
        ctypes.byref(gr) if gr is not None else None, _ptr(ws), ws.numel(), _stream(stream)))


def pa_slice_aggregate_w(dims, x, G, sp, num, den, S, W, ws, stream=None):
    d = _shapes(dims)
    _check_struct(sp, dims)
    _check(load().pa_slice_aggregate_w(ctypes.byref(dims), _arg(x, *d["x"], "x"), _arg(G, *d["G"], "G"),
                                       ctypes.byref(sp), _arg(num, *d["MC"], "num"),
                                       _arg(den, *d["M"], "den"), _arg(S, *d["MC"], "S"), _arg(W, *d["G"], "W"),
                                       _ptr(ws), ws.numel(), _stream(stream)))


def pa_slice_aggregate_noalloc(dims, x, G, sp, num, den, S, stream=None):
    """pa_slice_aggregate with the library's static scratch (no workspace)."""
    d = _shapes(dims)
    _check_struct(sp, dims)
    _check(load().pa_slice_aggregate_noalloc(ctypes.byref(dims), _arg(x, *d["x"], "x"),
                                             _arg(G, *d["G"], "G"), ctypes.byref(sp),
                                             _arg(num, *d["MC"], "num"), _arg(den, *d["M"], "den"),
                                             _arg(S, *d["MC"], "S"), _stream(stream)))


def pa_deslice_w(dims, W, Sp, y, ws, stream=None):
    d = _shapes(dims)
    _check(load().pa_deslice_w(ctypes.byref(dims), _arg(W, *d["G"], "W"), _arg(Sp, *d["MC"], "Sp"),
                               _arg(y, *d["x"], "y"), _ptr(ws), ws.numel(), _stream(stream)))


def pa_deslice_backward_w(dims, W, dY, dSp, ws, stream=None):
    d = _shapes(dims)
    _check(load().pa_deslice_backward_w(ctypes.byref(dims), _arg(W, *d["G"], "W"), _arg(dY, *d["x"], "dY"),
                                        _arg(dSp, *d["MC"], "dSp"), _ptr(ws), ws.numel(),
                                        _stream(stream)))


def pa_time_kernel(call: Optional[str], start=None, stop=None):
    """Arm (or, with call None, disarm) the kernel timing hook of this thread:
    ``start`` / ``stop`` are ``HipEvent`` objects."""
    _check(load().pa_time_kernel(call.encode() if call is not None else None,
                                 start.handle if start is not None else None,
                                 stop.handle if stop is not None else None))


def pa_stream_probe(dims, call: str, x, dY=None, G=None, out=None, stream=None):
    """One kernel moving the point tensors of ``call``'s streaming kernel
    with its loads and stores and no arithmetic (out receives x's rows)."""
    d = _shapes(dims)
    _check(load().pa_stream_probe(ctypes.byref(dims), call.encode(), _arg(x, *d["x"], "x"),
                                  _arg(dY, *d["x"], "dY") if dY is not None else None,
                                  _arg(G, *d["G"], "G") if G is not None else None,
                                  _arg(out, *d["x"], "out") if out is not None else None,
                                  _stream(stream)))


# HIP events straight from the HIP runtime (the library times its kernels on
# the caller's stream with these; torch.cuda.Event cannot be handed over).
HIP_EVENT_DISABLE_SYSTEM_FENCE = 0x20000000
_hip = None


def _hip_rt():
    global _hip
    if _hip is None:
        h = ctypes.CDLL("libamdhip64.so")
        h.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
        h.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        h.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                          ctypes.c_void_p]
        h.hipEventDestroy.argtypes = [ctypes.c_void_p]
        for f in ("hipEventCreateWithFlags", "hipEventRecord", "hipEventElapsedTime",
                  "hipEventDestroy"):
            getattr(h, f).restype = ctypes.c_int
        _hip = h
    return _hip


class HipEvent:
    """A timing HIP event.  By default it is recorded with a device-scope
    fence only (hipEventDisableSystemFence): no write-back of the caches to
    the host at each record, so timing a kernel disturbs the next one less."""

    def __init__(self, flags: int = HIP_EVENT_DISABLE_SYSTEM_FENCE):
        self.handle = ctypes.c_void_p()
        e = _hip_rt().hipEventCreateWithFlags(ctypes.byref(self.handle), flags)
        if e != 0:
            raise RuntimeError(f"hipEventCreateWithFlags failed ({e})")

    def record(self, stream=None):
        e = _hip_rt().hipEventRecord(self.handle, _stream(stream))
        if e != 0:
            raise RuntimeError(f"hipEventRecord failed ({e})")

    def elapsed_ms(self, end: "HipEvent") -> float:
        ms = ctypes.c_float()
        e = _hip_rt().hipEventElapsedTime(ctypes.byref(ms), self.handle, end.handle)
        if e != 0:
            raise RuntimeError(f"hipEventElapsedTime failed ({e})")
        return ms.value

    def __del__(self):
        if self.handle and _hip is not None:
            _hip.hipEventDestroy(self.handle)
            self.handle = ctypes.c_void_p()


# ---- block-stack primitives (include/pa.h) ----
def _nbytes(t) -> int:
    return 0 if t is None else t.numel() * t.element_size()


def _dt(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return PA_BF16
    if t.dtype == torch.float32:
        return PA_F32
    raise ValueError(f"unsupported dtype {t.dtype}")


def pa_gemm(A, B, D, transA=False, transB=False, alpha=1.0, beta=0.0, bias=None, ws=None,
            C=None, stream=None, prepare=False):
    """Row-major D = alpha op(A) op(B) + beta C (+ bias); C defaults to D.
    prepare: through pa_gemm_prepare (tunes the problem, synchronises)."""
    m = A.shape[1] if transA else A.shape[0]
    k = A.shape[0] if transA else A.shape[1]
    n = B.shape[0] if transB else B.shape[1]
    if (B.shape[1] if transB else B.shape[0]) != k:
        raise ValueError(f"pa_gemm: inner dimensions {k} and {tuple(B.shape)} do not match")
    dt = _dt(D)
    fn = load().pa_gemm_prepare if prepare else load().pa_gemm
    _check(fn(int(transA), int(transB), m, n, k, float(alpha), _ptr(A), _dt(A), _ptr(B), _dt(B),
              float(beta), _arg(C, m * n, dt, "C"), _arg(D, m * n, dt, "D"), dt,
              _arg(bias, n, PA_F32, "bias"), _ptr(ws), _nbytes(ws), _stream(stream)))


def pa_layernorm(x, y, mean, rstd, g=None, b=None, r=None, xs=None, eps=1e-5, stream=None):
    N, C = x.shape
    _check(load().pa_layernorm(N, C, float(eps), _dt(x), _ptr(x), _ptr(r), _ptr(xs), _ptr(g),
                               _ptr(b), _ptr(y), _ptr(mean), _ptr(rstd), _stream(stream)))


def pa_layernorm_backward(x, mean, rstd, dy, dx, g=None, dres=None, dg=None, db=None, ws=None,
                          stream=None):
    N, C = x.shape
    _check(load().pa_layernorm_backward(N, C, _dt(x), _ptr(x), _ptr(g), _ptr(mean), _ptr(rstd),
                                        _ptr(dy), _ptr(dres), _ptr(dx), _ptr(dg), _ptr(db),
                                        _ptr(ws), _nbytes(ws), _stream(stream)))


def pa_gelu(x, y, stream=None):
    n, dt = x.numel(), _dt(x)
    _check(load().pa_gelu(n, dt, _ptr(x), _arg(y, n, dt, "y"), _stream(stream)))


def pa_gelu_backward(x, dy, dx, stream=None):
    n, dt = x.numel(), _dt(x)
    _check(load().pa_gelu_backward(n, dt, _ptr(x), _arg(dy, n, dt, "dy"), _arg(dx, n, dt, "dx"),
                                   _stream(stream)))


def pa_mlp_up(X, W1, b1, G, ws, stream=None):
    """G [N,F] = GELU(X W1 + b1) in one kernel (bf16; X [N,K], W1 [K,F], b1
    [F] fp32); ws: a device buffer of at least 2 F K bytes."""
    N, K = X.shape
    F = W1.shape[1]
    _need(X, N * K, PA_BF16, "X")
    _check(load().pa_mlp_up(N, K, F, _ptr(X), _arg(W1, K * F, PA_BF16, "W1"),
                            _arg(b1, F, PA_F32, "b1"), _arg(G, N * F, PA_BF16, "G"), _ptr(ws),
                            _nbytes(ws), _stream(stream)))


def pa_mlp_up_backward(X, W1, b1, dY, W2, dU, ws, stream=None):
    """dU [N,F] = (dY W2^T) GELU'(X W1 + b1), the pre-activation recomputed
    (bf16; dY [N,K], W2 [F,K])."""
    N, K = X.shape
    F = W1.shape[1]
    _need(X, N * K, PA_BF16, "X")
    _check(load().pa_mlp_up_backward(N, K, F, _ptr(X), _arg(W1, K * F, PA_BF16, "W1"),
                                     _arg(b1, F, PA_F32, "b1"), _arg(dY, N * K, PA_BF16, "dY"),
                                     _arg(W2, F * K, PA_BF16, "W2"), _arg(dU, N * F, PA_BF16, "dU"),
                                     _ptr(ws), _nbytes(ws), _stream(stream)))


def pa_colsum(x, out, ws, stream=None):
    N, C = x.shape
    _check(load().pa_colsum(N, C, _dt(x), _ptr(x), _ptr(out), _ptr(ws), _nbytes(ws),
                            _stream(stream)))


def pa_project_fold(dims, Wp, bp, A, b, a, A_out, b_out, a_out, b_t_out, stream=None):
    _check(load().pa_project_fold(ctypes.byref(dims), _ptr(Wp), _ptr(bp), _ptr(A), _ptr(b),
                                  _ptr(a), _ptr(A_out), _ptr(b_out), _ptr(a_out), _ptr(b_t_out),
                                  _stream(stream)))


def pa_project_states(dims, S, Wp, bp, S_proj, stream=None):
    _check(load().pa_project_states(ctypes.byref(dims), _ptr(S), _ptr(Wp), _ptr(bp),
                                    _ptr(S_proj), _stream(stream)))


def pa_project_backward(dims, Wp, bp, A, a, S, dS_proj, folded, dWp, dbp, dS, gr, stream=None):
    _check(load().pa_project_backward(ctypes.byref(dims), _ptr(Wp), _ptr(bp), _ptr(A), _ptr(a),
                                      _ptr(S), _ptr(dS_proj), ctypes.byref(folded), _ptr(dWp),
                                      _ptr(dbp), _ptr(dS), ctypes.byref(gr), _stream(stream)))



# ---- per-head slicing layout (include/pa.h) ----
def pa_heads_relayout(src, dst, H, to_heads, stream=None):
    """[R,H,D] -> [H,R,D] (to_heads) or back; src/dst shapes (R, H*D) and
    (H, R, D), either way round."""
    if to_heads:
        R, C = src.shape
        assert dst.numel() == src.numel()
    else:
        R, C = dst.shape
        assert src.numel() == dst.numel()
    _check(load().pa_heads_relayout(R, H, C // H, _dt(src), int(bool(to_heads)), _ptr(src),
                                    _ptr(dst), _stream(stream)))


def pa_heads_expand(src, dst, H, blockdiag, stream=None):
    L = src.shape[0] if blockdiag else src.numel()
    _check(load().pa_heads_expand(H, L, int(bool(blockdiag)), _ptr(src), _ptr(dst),
                                  _stream(stream)))


def pa_heads_sum(src, dst, H, blockdiag, stream=None):
    L = dst.shape[0] if blockdiag else dst.numel()
    _check(load().pa_heads_sum(H, L, int(bool(blockdiag)), _ptr(src), _ptr(dst),
                               _stream(stream)))


def pa_heads_sum_batch(items, H, stream=None):
    """items: (src, dst, blockdiag) triples, each summed as pa_heads_sum
    would, all in one launch."""
    arr = (pa_heads_sum_item * len(items))()
    for i, (src, dst, bd) in enumerate(items):
        L = dst.shape[0] if bd else dst.numel()
        n = H * L * L if bd else H * L
        _need(src, n, PA_F32, "src")
        _need(dst, L * L if bd else L, PA_F32, "dst")
        arr[i] = pa_heads_sum_item(_ptr(src), _ptr(dst), L, int(bool(bd)))
    _check(load().pa_heads_sum_batch(H, len(items), arr, _stream(stream)))


# ---- per-head slicing in one launch per kernel (include/pa.h) ----
def make_heads_params(A, b=None, a=None, b_t=None, shared=False) -> pa_heads_params:
    """A [heads,D,M] (or [D,M] with shared) etc.; b_t a device fp32 tensor
    [heads] (or [1] with shared)."""
    sh = bool(shared)
    return _with(pa_heads_params(_ptr(A), _ptr(b), _ptr(a), _ptr(b_t), int(sh)),
                 A=(A, "CM" if sh else "hCM"), b=(b, "M" if sh else "hM"),
                 a=(a, "C" if sh else "hC"), b_t=(b_t, "1" if sh else "h"))


def pa_heads_workspace_size(dims, heads: int) -> int:
    n = ctypes.c_size_t(0)
    _check(load().pa_heads_workspace_size(ctypes.byref(dims), heads, ctypes.byref(n)))
    return n.value


def heads_workspace(dims, heads: int, device="cuda"):
    import torch
    return torch.empty(pa_heads_workspace_size(dims, heads), dtype=torch.uint8, device=device)


def pa_heads_slice_aggregate(dims, heads, x, G, hp, num, den, S, ws, stream=None):
    d = _shapes(dims, heads)
    _check_struct(hp, dims, heads)
    _check(load().pa_heads_slice_aggregate(ctypes.byref(dims), heads, _arg(x, *d["x"], "x"),
                                           _arg(G, *d["G"], "G"), ctypes.byref(hp),
                                           _arg(num, *d["MC"], "num"), _arg(den, *d["M"], "den"),
                                           _arg(S, *d["MC"], "S"), _ptr(ws), ws.numel(),
                                           _stream(stream)))


def pa_heads_deslice(dims, heads, x, G, hp, Sp, y, ws, stream=None):
    d = _shapes(dims, heads)
    _check_struct(hp, dims, heads)
    _check(load().pa_heads_deslice(ctypes.byref(dims), heads, _arg(x, *d["x"], "x"), _arg(G, *d["G"], "G"),
                                   ctypes.byref(hp), _arg(Sp, *d["MC"], "Sp"), _arg(y, *d["x"], "y"),
                                   _ptr(ws), ws.numel(), _stream(stream)))


def pa_heads_deslice_backward(dims, heads, x, G, hp, dY, dSp, ws, stream=None):
    d = _shapes(dims, heads)
    _check_struct(hp, dims, heads)
    _check(load().pa_heads_deslice_backward(ctypes.byref(dims), heads, _arg(x, *d["x"], "x"),
                                            _arg(G, *d["G"], "G"), ctypes.byref(hp),
                                            _arg(dY, *d["x"], "dY"), _arg(dSp, *d["MC"], "dSp"), _ptr(ws),
                                            ws.numel(), _stream(stream)))


def pa_heads_slice_aggregate_backward(dims, heads, x, G, hp, num, den, dS, Sp, dY, dx, gr, ws,
                                      stream=None):
    d = _shapes(dims, heads)
    _check_struct(hp, dims, heads)
    _check_struct(gr, dims, heads, stacked=True)
    _check(load().pa_heads_slice_aggregate_backward(
        ctypes.byref(dims), heads, _arg(x, *d["x"], "x"), _arg(G, *d["G"], "G"), ctypes.byref(hp),
        _arg(num, *d["MC"], "num"), _arg(den, *d["M"], "den"), _arg(dS, *d["MC"], "dS"), _arg(Sp, *d["MC"], "Sp"),
        _arg(dY, *d["x"], "dY"), _arg(dx, *d["x"], "dx"), ctypes.byref(gr), _ptr(ws), ws.numel(),
        _stream(stream)))

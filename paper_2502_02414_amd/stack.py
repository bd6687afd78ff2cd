"""A stack of Transolver++ blocks, forward and backward, through the C ABI.

A block is the Transformer block with Physics-Attention in place of
attention (Section 3; the block diagram of Figure 2a), read as pre-norm with
residual adds:

    x1 = x + PA(LN1(x)),    x2 = x1 + GELU(LN2(x1) W1 + b1) W2 + b2,

where PA starts with Algorithm 1's Project step x_proj = h Wp + bp.  The
Project step is folded: the slice parameters become A' = Wp A, b' = b + bp A,
a' = Wp a, b_t' = b_t + bp.a (pa_project_fold), the layer's streaming calls
run on h = LN1(x), and the states are projected, S_proj = S Wp + bp
(pa_project_states), before the token attention (whose optional Wo, bo is
the layer's output projection).  x_proj is never formed.

Every step is a call of libpa.so (the layer's calls, LayerNorm with the
residual add fused, the Project folding, the MLP's first product with its
GELU as one kernel (bf16; fp32 storage: a hipBLASLt GEMM and the GELU
kernel), and hipBLASLt GEMMs for the rest of the MLP, whose second GEMM
adds the residual).  torch only allocates the device buffers.  Per layer the
forward keeps x, LN1(x), x1, LN2(x1), GELU(u) (the backward's weight
gradient of W2 reads it) and the small per-layer state for the backward;
the pre-activation u is recomputed by the backward's fused kernel from
LN2(x1) (bf16; fp32 storage keeps u).

Parameters per layer (dict of device tensors): fp32 ln1_g, ln1_b, Wp [C,C],
bp [C], A [C,M], b [M], a [C], Wq, bq, Wk, bk, Wv, bv (optional Wo, bo),
ln2_g, ln2_b, b1 [4C], b2 [C]; W1 [C,4C] and W2 [4C,C] in the storage dtype;
plus the float b_t.
"""
from __future__ import annotations

from . import binding as B

ATTN = ("Wq", "bq", "Wk", "bk", "Wv", "bv", "Wo", "bo")


class BlockStack:
    def __init__(self, N, C, H, M, params, dtype, tau0=0.5, tau_min=0.01, eps=1e-5,
                 ln_eps=1e-5, device="cuda"):
        import torch
        self.torch = torch
        self.N, self.C, self.H, self.M = N, C, H, M
        self.params = params
        self.dt = dtype                       # torch dtype of the point-side tensors
        self.pdt = B.PA_BF16 if dtype == torch.bfloat16 else B.PA_F32
        self.ln_eps = ln_eps
        self.dims = B.make_dims(N, C, H, M, tau0, tau_min, eps, self.pdt)
        self.ws = B.workspace(self.dims, device)
        # scratch of the sums over rows (LayerNorm gains, bias gradients) and of hipBLASLt
        self.ws_rows = torch.empty(1024 * 4 * C, dtype=torch.float32, device=device)
        self.ws_gemm = torch.empty(256 << 20, dtype=torch.uint8, device=device)
        self.tuned = set()  # GEMM problems already tuned (pa_gemm_prepare)
        # bf16: the MLP's first product and GELU as one kernel (pa_mlp_up)
        self.fused_mlp = self.pdt == B.PA_BF16 and C in (64, 128, 256)
        self.dev = device

    # -- helpers ------------------------------------------------------------
    def _e(self, *shape, dt=None):
        return self.torch.empty(*shape, dtype=dt or self.dt, device=self.dev)

    def _f(self, *shape):
        return self.torch.empty(*shape, dtype=self.torch.float32, device=self.dev)

    def _gemm(self, A, Bm, D, **kw):
        # each GEMM problem is tuned once, on its first call (pa_gemm_prepare
        # synchronises); later calls never synchronise
        key = (tuple(A.shape), A.dtype, tuple(Bm.shape), Bm.dtype, D.dtype,
               tuple(sorted((k, v if isinstance(v, (bool, float, int)) else v is not None)
                            for k, v in kw.items())))
        first = key not in self.tuned
        self.tuned.add(key)
        B.pa_gemm(A, Bm, D, ws=self.ws_gemm, prepare=first, **kw)

    def _folded(self, p):
        """The folded slice parameters of a layer (pa_project_fold)."""
        C, M = self.C, self.M
        A_f, a_f = self._e(C, M), self._e(C)
        b_f, bt_f = self._f(M), self._f(1)
        B.pa_project_fold(self.dims, p["Wp"], p["bp"], p["A"], p.get("b"), p.get("a"), A_f, b_f,
                          a_f, bt_f)
        sp = B.make_slice_params(A_f, b_f, a_f, p.get("b_t", 0.0), b_t_dev=bt_f)
        return {"A": A_f, "b": b_f, "a": a_f, "bt": bt_f, "sp": sp}

    # -- forward ------------------------------------------------------------
    def forward(self, x, Gs):
        """x [N,C] (storage dtype), Gs: one Gumbel tensor [N,M] (or None) per
        layer.  Returns the output [N,C]; keeps what the backward needs."""
        N, C, M = self.N, self.C, self.M
        self.caches = []
        for p, G in zip(self.params, Gs):
            c = {"x": x, "G": G}
            h, m1, r1 = self._e(N, C), self._f(N), self._f(N)
            B.pa_layernorm(x, h, m1, r1, g=p["ln1_g"], b=p["ln1_b"], eps=self.ln_eps)
            fo = self._folded(p)
            num, den, S, S_proj, Sp = self._f(M, C), self._f(M), self._f(M, C), self._f(M, C), \
                self._f(M, C)
            B.pa_slice_aggregate(self.dims, h, G, fo["sp"], num, den, S, self.ws)
            B.pa_project_states(self.dims, S, p["Wp"], p["bp"], S_proj)
            apr = B.make_attn_params(**{k: p[k] for k in ATTN if p.get(k) is not None})
            B.pa_token_attention(self.dims, S_proj, apr, Sp, self.ws)
            y = self._e(N, C)
            B.pa_deslice(self.dims, h, G, fo["sp"], Sp, y, self.ws)
            # x1 = x + y (the first residual add) fused into LN2
            x1, h2, m2, r2 = self._e(N, C), self._e(N, C), self._f(N), self._f(N)
            B.pa_layernorm(x, h2, m2, r2, g=p["ln2_g"], b=p["ln2_b"], r=y, xs=x1, eps=self.ln_eps)
            del y
            gu = self._e(N, 4 * C)
            if self.fused_mlp:
                # GELU(h2 W1 + b1) in one kernel; u is recomputed in the backward
                u = None
                B.pa_mlp_up(h2, p["W1"], p["b1"], gu, self.ws_gemm)
            else:
                u = self._e(N, 4 * C)
                self._gemm(h2, p["W1"], u, bias=p["b1"])
                B.pa_gelu(u, gu)
            x2 = self._e(N, C)
            # x2 = x1 + GELU(u) W2 + b2 (the second residual add in the GEMM)
            self._gemm(gu, p["W2"], x2, bias=p["b2"], beta=1.0, C=x1)
            c.update({"h": h, "m1": m1, "r1": r1, "fold": fo, "num": num, "den": den, "S": S,
                      "S_proj": S_proj, "Sp": Sp, "apr": apr, "x1": x1, "h2": h2, "m2": m2,
                      "r2": r2, "u": u, "gu": gu})
            self.caches.append(c)
            x = x2
        return x

    # -- backward -----------------------------------------------------------
    def backward(self, dy):
        """dy [N,C]: the gradient of the stack's output.  Returns (dx,
        [grads per layer]) with fp32 parameter gradients named d<param>."""
        N, C, M = self.N, self.C, self.M
        grads = [None] * len(self.params)
        for l in reversed(range(len(self.params))):
            p, c = self.params[l], self.caches[l]
            g = {}
            # MLP: x2 = x1 + GELU(u) W2 + b2
            gu = c.pop("gu")                                       # GELU(u), kept by the forward
            g["dW2"] = self._f(4 * C, C)
            self._gemm(gu, dy, g["dW2"], transA=True)
            g["db2"] = self._f(C)
            B.pa_colsum(dy, g["db2"], self.ws_rows)
            if self.fused_mlp:                                     # du, in place of gu
                B.pa_mlp_up_backward(c["h2"], p["W1"], p["b1"], dy, p["W2"], gu, self.ws_gemm)
            else:
                self._gemm(dy, p["W2"], gu, transB=True)          # dGELU(u), in place of gu
                B.pa_gelu_backward(c["u"], gu, gu)                 # du
            g["dW1"] = self._f(C, 4 * C)
            self._gemm(c["h2"], gu, g["dW1"], transA=True)
            g["db1"] = self._f(4 * C)
            B.pa_colsum(gu, g["db1"], self.ws_rows)
            dh2 = self._e(N, C)
            self._gemm(gu, p["W1"], dh2, transB=True)
            del gu
            dx1 = self._e(N, C)
            g["dln2_g"], g["dln2_b"] = self._f(C), self._f(C)
            B.pa_layernorm_backward(c["x1"], c["m2"], c["r2"], dh2, dx1, g=p["ln2_g"], dres=dy,
                                    dg=g["dln2_g"], db=g["dln2_b"], ws=self.ws_rows)
            del dh2
            # Physics-Attention on h with the folded Project step; dY = dx1
            fo = c["fold"]
            dSp, dS_proj = self._f(M, C), self._f(M, C)
            B.pa_deslice_backward(self.dims, c["h"], c["G"], fo["sp"], dx1, dSp, self.ws)
            ag = {k: self._f(C, C) for k in ("dWq", "dWk", "dWv")}
            ag.update({k: self._f(C) for k in ("dbq", "dbk", "dbv")})
            if p.get("Wo") is not None:
                ag["dWo"], ag["dbo"] = self._f(C, C), self._f(C)
            B.pa_token_attention_backward(self.dims, c["S_proj"], c["apr"], dSp, dS_proj,
                                          B.make_attn_grads(**ag), self.ws)
            g.update(ag)
            dS = self._f(M, C)
            self._gemm(dS_proj, p["Wp"], dS, transB=True)         # dS = dS_proj Wp^T
            gf = {"dA": self._f(C, M), "db": self._f(M), "da": self._f(C), "db_t": self._f(1),
                  "dtau0": self._f(1)}
            dh = self._e(N, C)
            B.pa_slice_aggregate_backward(self.dims, c["h"], c["G"], fo["sp"], c["num"], c["den"],
                                          dS, c["Sp"], dx1, dh, B.make_slice_grads(**gf), self.ws)
            g["dWp"], g["dbp"] = self._f(C, C), self._f(C)
            g.update({"dA": self._f(C, M), "db": self._f(M), "da": self._f(C),
                      "db_t": self._f(1)})
            B.pa_project_backward(self.dims, p["Wp"], p["bp"], p["A"], p.get("a"), c["S"], dS_proj,
                                  B.make_slice_grads(**gf), g["dWp"], g["dbp"], None,
                                  B.make_slice_grads(dA=g["dA"], db=g["db"], da=g["da"],
                                                     db_t=g["db_t"]))
            # LN1 and the first residual: dx = LN1'(dh) + dx1
            dx = self._e(N, C)
            g["dln1_g"], g["dln1_b"] = self._f(C), self._f(C)
            B.pa_layernorm_backward(c["x"], c["m1"], c["r1"], dh, dx, g=p["ln1_g"], dres=dx1,
                                    dg=g["dln1_g"], db=g["dln1_b"], ws=self.ws_rows)
            grads[l] = g
            dy = dx
        return dy, grads

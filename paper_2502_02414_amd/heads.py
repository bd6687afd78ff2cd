"""Per-head sliced Physics-Attention layer, forward and backward, through the C ABI.

Per-head slicing carries the heads of Eq. 2 into the slicing of Eq. 1: the
C channels split into H contiguous blocks of D = C/H; head h slices its own
block x_h [N,D] with its own slice parameters (A_h [D,M], b_h, Ada-Temp a_h,
b_t,h; Eq. 3) and Gumbel noise G_h [N,M] (Eq. 4), forms its own M states
S_h [M,D] (Eq. 1), runs one-head attention of width D among them with the
token projections shared by the heads (Eq. 2's Linear acting on the last
axis of the [H,M,D] states), and deslices W_h S'_h into its own block.  With
G = None and a = None it is the Transolver mode (no noise, constant
temperature tau0 + b_t).  The slice parameters may also be one set for all
heads (A given as [D,M]); their gradients are then summed over the heads.

Layout: the point-side tensors are head-major, x, G, dY, y, dx [H,N,D]
(G [H,N,M]), so a head's rows are contiguous; pa_heads_relayout moves a
[N,C] tensor to and from it.  Each head runs the layer's streaming calls
(dims with C = D, H = 1).  The token attention of all heads is one
pa_token_attention call (dims with C = H D, H heads) on the states side by
side, [M, H D], with the shared D x D projections laid on the block
diagonal (pa_heads_expand): head h's query is then S_h Wq + bq, and its
attention runs over its own M tokens only.  The token gradients are the
sums of the diagonal blocks (pa_heads_sum).  Every step is a call of
libpa.so; torch only allocates the device buffers.

Launches: by default (M a multiple of 8, at most 16 heads) each phase is
ONE pa_heads_* call, whose table, streaming and reduction kernels each cover
all heads in one launch (the head is the grid's second index).  Otherwise
(or with batched=False) each head makes its own one-head call, and the heads
of a phase are spread over `streams` streams (default priority, forked from
and joined back into the caller's current stream by events), each with its
own workspace, so that one head's small kernels overlap another head's
streaming pass.  Every head's arithmetic, and the order of its sums, is the
same either way: the results are the same bits.

Parameters (dict of device tensors): A [H,D,M] or [D,M] and a [H,D] or [D]
in the storage dtype (a nullable), b [H,M] or [M] fp32 (nullable), b_t a
list of H floats or one float; Wq, Wk, Wv [D,D], bq, bk, bv [D] fp32
(optional Wo [D,D], bo [D]).  M a multiple of 4 when b is per head.
"""
from __future__ import annotations

from . import binding as B

ATTN_W = ("Wq", "Wk", "Wv", "Wo")
ATTN_B = ("bq", "bk", "bv", "bo")


class HeadSlicedLayer:
    def __init__(self, N, H, D, M, params, dtype, tau0=0.5, tau_min=0.01, eps=1e-5,
                 device="cuda", streams=2, batched=None):
        import torch
        self.torch = torch
        self.N, self.H, self.D, self.M, self.C = N, H, D, M, H * D
        self.dt = dtype
        pdt = B.PA_BF16 if dtype == torch.bfloat16 else B.PA_F32
        self.dev = device
        self.shared = params["A"].dim() == 2
        if not self.shared and params.get("b") is not None and M % 4:
            raise ValueError("per-head biases b [H,M] need M to be a multiple of 4")
        self.dims_h = B.make_dims(N, D, 1, M, tau0, tau_min, eps, pdt)
        self.dims_t = B.make_dims(N, H * D, H, M, tau0, tau_min, eps, pdt)
        self.batched = (M % 8 == 0 and H <= 16) if batched is None else bool(batched)
        if self.batched and (M % 8 or H > 16):
            raise ValueError("batched per-head calls need M a multiple of 8 and H <= 16")
        self.ws_b = B.heads_workspace(self.dims_h, H, device) if self.batched else None
        self.ns = 1 if self.batched else max(1, min(int(streams), H))
        self.ws_h = [] if self.batched else [B.workspace(self.dims_h, device)
                                             for _ in range(self.ns)]
        self.side = [torch.cuda.Stream(device=device) for _ in range(self.ns - 1)]
        self.ws_t = B.workspace(self.dims_t, device)
        self.set_params(params)

    def _f(self, *shape):
        return self.torch.empty(*shape, dtype=self.torch.float32, device=self.dev)

    def set_params(self, p):
        """Per-head slice parameter structs and the block-diagonal token
        projections of the H-head call (after every parameter update)."""
        self.p = p
        H, C = self.H, self.C
        bt = p.get("b_t", 0.0)
        self.sp = []
        for h in range(H):
            pick = (lambda k: p.get(k)) if self.shared else \
                (lambda k: None if p.get(k) is None else p[k][h])
            b_t = float(bt) if self.shared or isinstance(bt, (int, float)) else float(bt[h])
            self.sp.append(B.make_slice_params(pick("A"), pick("b"), pick("a"), b_t))
        bts = [float(bt)] if self.shared or isinstance(bt, (int, float)) else [float(v) for v in bt]
        if not self.shared and len(bts) == 1:
            bts = bts * H
        self.bt_dev = self.torch.tensor(bts, dtype=self.torch.float32, device=self.dev)
        self.hp = B.make_heads_params(p["A"], p.get("b"), p.get("a"), self.bt_dev,
                                      shared=self.shared)
        self.att = {}
        for k in ATTN_W:
            if p.get(k) is not None:
                self.att[k] = self._f(C, C)
                B.pa_heads_expand(p[k], self.att[k], H, blockdiag=True)
        for k in ATTN_B:
            if p.get(k) is not None:
                self.att[k] = self._f(C)
                B.pa_heads_expand(p[k], self.att[k], H, blockdiag=False)
        self.ap = B.make_attn_params(**self.att)

    def _heads(self, fn):
        """fn(h, ws, stream) for every head, head h on stream h mod ns (the
        current stream and the side streams), joined back into the current
        stream."""
        torch = self.torch
        main = torch.cuda.current_stream()
        if self.ns > 1:
            fork = torch.cuda.Event()
            fork.record(main)
            for st in self.side:
                st.wait_event(fork)
        for h in range(self.H):
            k = h % self.ns
            fn(h, self.ws_h[k], main if k == 0 else self.side[k - 1])
        if self.ns > 1:
            for st in self.side:
                done = torch.cuda.Event()
                done.record(st)
                main.wait_event(done)

    # -- layout helpers -----------------------------------------------------
    def to_heads(self, x):
        """[N,C] -> head-major [H,N,D]."""
        out = self.torch.empty(self.H, x.shape[0], self.D, dtype=x.dtype, device=self.dev)
        B.pa_heads_relayout(x, out, self.H, to_heads=True)
        return out

    def from_heads(self, xh):
        """Head-major [H,N,D] -> [N,C]."""
        out = self.torch.empty(xh.shape[1], self.C, dtype=xh.dtype, device=self.dev)
        B.pa_heads_relayout(xh, out, self.H, to_heads=False)
        return out

    # -- forward ------------------------------------------------------------
    def forward(self, xh, G=None):
        """xh [H,N,D], G [H,N,M] or None (storage dtype).  Returns y [H,N,D]."""
        H, N, D, M, C = self.H, self.N, self.D, self.M, self.C
        g = (lambda h: None) if G is None else (lambda h: G[h])
        num, den, S_h = self._f(H, M, D), self._f(H, M), self._f(H, M, D)
        if self.batched:
            B.pa_heads_slice_aggregate(self.dims_h, H, xh, G, self.hp, num, den, S_h, self.ws_b)
        else:
            self._heads(lambda h, ws, st: B.pa_slice_aggregate(
                self.dims_h, xh[h], g(h), self.sp[h], num[h], den[h], S_h[h], ws, stream=st))
        S = self._f(M, C)
        B.pa_heads_relayout(S_h, S, H, to_heads=False)
        Sp = self._f(M, C)
        B.pa_token_attention(self.dims_t, S, self.ap, Sp, self.ws_t)
        Sp_h = self._f(H, M, D)
        B.pa_heads_relayout(Sp, Sp_h, H, to_heads=True)
        yh = self.torch.empty(H, N, D, dtype=xh.dtype, device=self.dev)
        if self.batched:
            B.pa_heads_deslice(self.dims_h, H, xh, G, self.hp, Sp_h, yh, self.ws_b)
        else:
            self._heads(lambda h, ws, st: B.pa_deslice(
                self.dims_h, xh[h], g(h), self.sp[h], Sp_h[h], yh[h], ws, stream=st))
        self.cache = {"x": xh, "G": G, "num": num, "den": den, "S": S, "Sp_h": Sp_h}
        return yh

    # -- backward -----------------------------------------------------------
    def backward(self, dYh):
        """dYh [H,N,D].  Returns (dx [H,N,D], grads): fp32 gradients named
        d<param>; the slice parameters' per head ([H,...]; db_t [H]) or
        summed when shared, the token projections' and dtau0 summed over the
        heads."""
        H, N, D, M, C = self.H, self.N, self.D, self.M, self.C
        c = self.cache
        xh, G = c["x"], c["G"]
        g = (lambda h: None) if G is None else (lambda h: G[h])
        dSp_h = self._f(H, M, D)
        if self.batched:
            B.pa_heads_deslice_backward(self.dims_h, H, xh, G, self.hp, dYh, dSp_h, self.ws_b)
        else:
            self._heads(lambda h, ws, st: B.pa_deslice_backward(
                self.dims_h, xh[h], g(h), self.sp[h], dYh[h], dSp_h[h], ws, stream=st))
        dSp = self._f(M, C)
        B.pa_heads_relayout(dSp_h, dSp, H, to_heads=False)
        ag = {"d" + k: self._f(C, C) for k in ATTN_W if k in self.att}
        ag.update({"d" + k: self._f(C) for k in ATTN_B if k in self.att})
        dS = self._f(M, C)
        B.pa_token_attention_backward(self.dims_t, c["S"], self.ap, dSp, dS,
                                      B.make_attn_grads(**ag), self.ws_t)
        dS_h = self._f(H, M, D)
        B.pa_heads_relayout(dS, dS_h, H, to_heads=True)
        per = {"dA": self._f(H, D, M), "db": self._f(H, M), "da": self._f(H, D),
               "db_t": self._f(H), "dtau0": self._f(H)}
        dxh = self.torch.empty(H, N, D, dtype=xh.dtype, device=self.dev)
        if self.batched:
            B.pa_heads_slice_aggregate_backward(self.dims_h, H, xh, G, self.hp, c["num"], c["den"],
                                                dS_h, c["Sp_h"], dYh, dxh,
                                                B.make_slice_grads(**per), self.ws_b)
        else:
            grs = [B.make_slice_grads(**{k: v[h] for k, v in per.items()}) for h in range(H)]
            self._heads(lambda h, ws, st: B.pa_slice_aggregate_backward(
                self.dims_h, xh[h], g(h), self.sp[h], c["num"][h], c["den"][h], dS_h[h],
                c["Sp_h"][h], dYh[h], dxh[h], grs[h], ws, stream=st))
        # the shared parameters' gradients: sums over the heads, up to eight
        # per launch (pa_heads_sum_batch)
        grads, sums = {}, []
        for k in ATTN_W:
            if "d" + k in ag:
                grads["d" + k] = self._f(D, D)
                sums.append((ag["d" + k], grads["d" + k], True))
        for k in ATTN_B:
            if "d" + k in ag:
                grads["d" + k] = self._f(D)
                sums.append((ag["d" + k], grads["d" + k], False))
        grads["dtau0"] = self._f(1)
        sums.append((per["dtau0"], grads["dtau0"], False))
        for k in ("dA", "db", "da", "db_t"):
            if self.shared:
                shape = per[k].shape[1:] or (1,)
                grads[k] = self._f(*shape)
                sums.append((per[k], grads[k], False))
            else:
                grads[k] = per[k]
        for i in range(0, len(sums), 8):
            B.pa_heads_sum_batch(sums[i:i + 8], H)
        return dxh, grads

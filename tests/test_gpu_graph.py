"""The layer's call sequence captured in a HIP graph (torch.cuda.CUDAGraph on
the caller's stream) and replayed: every call of the library only launches
kernels on the stream it is given (no allocation, copy, memset or wait), so
a replay must give the eager results bit for bit.  The graph is replayed
several times with eager work and synchronisations between replays, and
every replay is compared with the eager run."""
import numpy as np
import pytest

from paper_2502_02414_amd import binding as B
from pa_cases import Gpu, host, make_case, say

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dt,N,C,H,M", [("f32", 4096, 64, 4, 16), ("bf16", 32768, 256, 8, 32)])
def test_layer_graph_replays_match_eager(dt, N, C, H, M):
    import torch
    say(f"graph {dt} N={N} C={C} H={H} M={M}")
    g = Gpu(make_case(N, C, H, M, dt, biases=True))
    f32 = lambda *s: torch.zeros(*s, dtype=torch.float32, device="cuda")
    num, den, S, Sp, dSp, dS = f32(M, C), f32(M), f32(M, C), f32(M, C), f32(M, C), f32(M, C)
    y = torch.zeros(N, C, dtype=g.x.dtype, device="cuda")
    dx = torch.zeros_like(y)
    ag = {k: f32(C, C) for k in ("dWq", "dWk", "dWv")}
    ag.update({k: f32(C) for k in ("dbq", "dbk", "dbv")})
    sg = {"dA": f32(C, M), "db": f32(M), "da": f32(C), "db_t": f32(1), "dtau0": f32(1)}
    agr, sgr = B.make_attn_grads(**ag), B.make_slice_grads(**sg)
    outs = {"num": num, "den": den, "S": S, "Sp": Sp, "y": y, "dSp": dSp, "dS": dS, "dx": dx}
    outs.update(ag)
    outs.update(sg)

    def step():
        B.pa_slice_aggregate(g.dims, g.x, g.G, g.sp, num, den, S, g.ws)
        B.pa_token_attention(g.dims, S, g.ap, Sp, g.ws)
        B.pa_deslice(g.dims, g.x, g.G, g.sp, Sp, y, g.ws)
        B.pa_deslice_backward(g.dims, g.x, g.G, g.sp, g.dY, dSp, g.ws)
        B.pa_token_attention_backward(g.dims, S, g.ap, dSp, dS, agr, g.ws)
        B.pa_slice_aggregate_backward(g.dims, g.x, g.G, g.sp, num, den, dS, Sp, g.dY, dx, sgr,
                                      g.ws)

    step()
    torch.cuda.synchronize()
    eager = {k: host(v).copy() for k, v in outs.items()}
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):   # warm-up on the capture stream
        step()
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    for rep in range(3):
        for v in outs.values():     # eager work between replays: clear the outputs
            v.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for k, v in outs.items():
            np.testing.assert_array_equal(host(v), eager[k], err_msg=f"replay {rep}: {k}")
    say("  3 replays equal the eager run")

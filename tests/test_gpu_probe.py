"""The stream probe (pa_stream_probe): one kernel that moves a streaming
pass's point tensors exactly as that pass's kernel does and computes
nothing.  Its output rows are the rows of x, so the test checks them bit
for bit (every row of a ragged N, every channel of a row narrower than the
kernel's width), and that the read-only passes run."""
import pytest

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("N,C,M,dt", [(1001, 256, 32, "bf16"), (777, 48, 20, "bf16"),
                                      (513, 96, 64, "f32"), (2500, 256, 64, "bf16")])
def test_probe_moves_the_rows(N, C, M, dt):
    import torch
    from paper_2502_02414_amd import binding as B
    t = torch.bfloat16 if dt == "bf16" else torch.float32
    g = torch.Generator(device="cuda").manual_seed(N + C)
    x = torch.randn(N, C, device="cuda", generator=g).to(t)
    dY = torch.randn(N, C, device="cuda", generator=g).to(t)
    G = torch.randn(N, M, device="cuda", generator=g).to(t)
    dims = B.make_dims(N, C, max(1, C // 16), M, 0.5, 0.01, 1e-5,
                       B.PA_BF16 if dt == "bf16" else B.PA_F32)
    for call in ("pa_deslice", "pa_slice_aggregate_backward"):
        out = torch.full((N, C), float("nan"), device="cuda").to(t)
        B.pa_stream_probe(dims, call, x, dY if "backward" in call else None, G, out)
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16 if dt == "bf16" else torch.int32),
                           x.view(torch.int16 if dt == "bf16" else torch.int32)), call
    for call in ("pa_slice_aggregate", "pa_deslice_backward"):
        B.pa_stream_probe(dims, call, x, dY if "backward" in call else None, G)
        B.pa_stream_probe(dims, call, x, dY if "backward" in call else None, None)
    torch.cuda.synchronize()

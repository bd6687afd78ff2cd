"""pa_slice_aggregate_noalloc (the library's static scratch, no workspace)
against pa_slice_aggregate (a caller's workspace), through the C ABI: the
same kernels in the same launch shapes, so the outputs must be identical bit
for bit, and within the parity bar of the oracle.  Calls in a row share the
device's one scratch array: a large call, then smaller ones of other shapes,
each checked."""
import numpy as np
import pytest

from paper_2502_02414_amd import binding as B
from pa_cases import TOL, Gpu, host, make_case, oracle_layer, rel_l2, say

pytestmark = pytest.mark.gpu

# (N, C, H, M, dtype): the bench's layer shape at 66k points first, then
# smaller inputs and other shapes (other table images and record sizes)
SEQUENCE = [(66013, 256, 8, 32, "bf16"), (3001, 256, 8, 32, "bf16"), (1000, 64, 4, 16, "f32"),
            (2049, 128, 8, 64, "f32")]


def test_noalloc_matches_workspace_call_twice_in_a_row():
    import torch
    for shape in SEQUENCE:
        say(f"noalloc {shape}")
        c = make_case(*shape)
        g = Gpu(c)
        num, den, S = g.aggregate()
        num2, den2, S2 = g.empty(c.M, c.C), g.empty(c.M), g.empty(c.M, c.C)
        B.pa_slice_aggregate_noalloc(g.dims, g.x, g.G, g.sp, num2, den2, S2)
        torch.cuda.synchronize()
        for k, a, b in (("num", num, num2), ("den", den, den2), ("S", S, S2)):
            assert torch.equal(a, b), (shape, k)
        f, _ = oracle_layer(c)
        for k, v in (("num", num2), ("den", den2), ("S", S2)):
            e = rel_l2(host(v), f[k])
            say(f"  {k:4s} rel_l2 = {e:.3e}  (bar {TOL[c.dt]:.0e})")
            assert e <= TOL[c.dt], (shape, k, e)


def test_noalloc_refuses_bad_arguments():
    c = make_case(100, 64, 4, 16, "f32")
    g = Gpu(c)
    num, den, S = g.empty(c.M, c.C), g.empty(c.M), g.empty(c.M, c.C)
    lib = B.load()
    import ctypes
    st = lib.pa_slice_aggregate_noalloc(ctypes.byref(g.dims), None, None, ctypes.byref(g.sp),
                                        num.data_ptr(), den.data_ptr(), S.data_ptr(), None)
    assert st == B.PA_ERR_INVALID and "x" in lib.pa_last_error().decode()

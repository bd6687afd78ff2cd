"""The C-ABI library loads, exports every symbol include/pa.h declares, and
rejects bad arguments on the host before launching anything.

These tests make no compute calls: every call below fails validation (or only
asks for the workspace size), so they run without a GPU.  The fake device
addresses are never dereferenced.
"""
import ctypes
import os
import re

import pytest

from paper_2502_02414_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(B.LIB_PATH):
        from paper_2502_02414_amd import build
        build.build()
    return B.load()


def _declared_symbols():
    with open(os.path.join(ROOT, "include", "pa.h")) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(pa_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(lib):
    declared = _declared_symbols()
    assert len(declared) == 38
    assert sorted(B.SYMBOLS) == declared
    for name in declared:
        assert hasattr(lib, name), name


def test_version(lib):
    assert lib.pa_version() == 8


def _dims(**kw):
    d = dict(N=1000, C=64, H=4, M=16, tau0=0.5, tau_min=0.01, eps=1e-5, dtype=B.PA_F32)
    d.update(kw)
    return B.make_dims(**d)


def _ws_size(lib, dims):
    n = ctypes.c_size_t(0)
    st = lib.pa_workspace_size(ctypes.byref(dims), ctypes.byref(n))
    return st, n.value


@pytest.mark.parametrize("kw,status", [
    (dict(N=0), B.PA_ERR_INVALID),
    (dict(M=0), B.PA_ERR_INVALID),
    (dict(M=65), B.PA_ERR_INVALID),
    (dict(H=3), B.PA_ERR_INVALID),
    (dict(tau_min=0.0), B.PA_ERR_INVALID),
    (dict(eps=-1.0), B.PA_ERR_INVALID),
    (dict(tau0=float("nan")), B.PA_ERR_INVALID),
    (dict(dtype=7), B.PA_ERR_INVALID),
    (dict(C=40, H=4), B.PA_ERR_UNSUPPORTED),
    (dict(C=512, H=8), B.PA_ERR_UNSUPPORTED),
    (dict(C=272, H=8), B.PA_ERR_UNSUPPORTED),
])
def test_dims_validation(lib, kw, status):
    st, _ = _ws_size(lib, _dims(**kw))
    assert st == status
    assert lib.pa_last_error().decode() != ""


@pytest.mark.parametrize("C", list(range(16, 257, 16)))
def test_every_multiple_of_16_channels_is_served(lib, C):
    # rows of C channels run on the kernels of the next width up (32, 64, 128
    # or 256) with zero table columns; the workspace holds that width's tables
    st, n = _ws_size(lib, _dims(C=C, H=16))
    assert st == B.PA_OK and n > 0


def test_workspace_size_grows_with_shape(lib):
    st1, n1 = _ws_size(lib, _dims())
    st2, n2 = _ws_size(lib, _dims(C=256, H=8, M=32, dtype=B.PA_BF16, N=1_000_000))
    assert st1 == st2 == B.PA_OK
    assert 0 < n1 < n2
    assert n2 < 64 << 20  # partial records and tables only: no O(N) scratch


FAKE = 0x7f0000000000  # aligned, never dereferenced


def _gpu_visible() -> bool:
    try:
        import torch
        return torch.cuda.device_count() > 0  # counts devices without initialising them
    except Exception:
        return False


# The calls below hand the library a fake device address and rely on host
# validation failing first; where a GPU could be reached, a regression in
# that validation would launch a kernel at it, so they run only without one.
fake_addresses = pytest.mark.skipif(_gpu_visible(),
                                    reason="fake device addresses only where no GPU is visible")


@fake_addresses
def test_null_and_misaligned_pointers_rejected(lib):
    d = _dims()
    sp = B.pa_slice_params(FAKE, None, None, 0.0)
    _, n = _ws_size(lib, d)
    # x missing
    st = lib.pa_slice_aggregate(ctypes.byref(d), None, None, ctypes.byref(sp), FAKE, FAKE, FAKE,
                                FAKE, n, None)
    assert st == B.PA_ERR_INVALID and "x" in lib.pa_last_error().decode()
    # misaligned x
    st = lib.pa_slice_aggregate(ctypes.byref(d), FAKE + 2, None, ctypes.byref(sp), FAKE, FAKE,
                                FAKE, FAKE, n, None)
    assert st == B.PA_ERR_INVALID and "aligned" in lib.pa_last_error().decode()
    # A missing
    sp0 = B.pa_slice_params(None, None, None, 0.0)
    st = lib.pa_deslice(ctypes.byref(d), FAKE, None, ctypes.byref(sp0), FAKE, FAKE, FAKE, n,
                        None)
    assert st == B.PA_ERR_INVALID
    # only one of Sp / dY
    st = lib.pa_slice_aggregate_backward(ctypes.byref(d), FAKE, None, ctypes.byref(sp), FAKE,
                                         FAKE, FAKE, FAKE, None, FAKE, None, FAKE, n, None)
    assert st == B.PA_ERR_INVALID and "both" in lib.pa_last_error().decode()


@fake_addresses
def test_small_workspace_rejected(lib):
    d = _dims()
    sp = B.pa_slice_params(FAKE, None, None, 0.0)
    _, n = _ws_size(lib, d)
    st = lib.pa_slice_aggregate(ctypes.byref(d), FAKE, None, ctypes.byref(sp), FAKE, FAKE, FAKE,
                                FAKE, n - 256, None)
    assert st == B.PA_ERR_WORKSPACE
    st = lib.pa_slice_aggregate(ctypes.byref(d), FAKE, None, ctypes.byref(sp), FAKE, FAKE, FAKE,
                                None, n, None)
    assert st == B.PA_ERR_WORKSPACE


@fake_addresses
def test_attention_argument_checks(lib):
    d = _dims()
    _, n = _ws_size(lib, d)
    ap = B.pa_attn_params(FAKE, None, None, None, FAKE, None, None, None)  # Wk missing
    st = lib.pa_token_attention(ctypes.byref(d), FAKE, ctypes.byref(ap), FAKE, FAKE, n, None)
    assert st == B.PA_ERR_INVALID and "Wk" in lib.pa_last_error().decode()
    ap = B.pa_attn_params(FAKE, None, FAKE, None, FAKE, None, None, FAKE)  # bo without Wo
    st = lib.pa_token_attention(ctypes.byref(d), FAKE, ctypes.byref(ap), FAKE, FAKE, n, None)
    assert st == B.PA_ERR_INVALID


@fake_addresses
def test_unserved_table_shape_is_unsupported(lib):
    # the backward tables of C=256, M=64 in fp32 exceed the 160 KB of LDS
    d = _dims(C=256, H=8, M=64, dtype=B.PA_F32)
    sp = B.pa_slice_params(FAKE, None, None, 0.0)
    _, n = _ws_size(lib, d)
    st = lib.pa_slice_aggregate_backward(ctypes.byref(d), FAKE, None, ctypes.byref(sp), FAKE,
                                         FAKE, FAKE, None, None, FAKE, None, FAKE, n, None)
    assert st == B.PA_ERR_UNSUPPORTED


@fake_addresses
def test_kernel_timing_hook_checks(lib):
    # host-only: arming records nothing until a call launches its kernel
    assert lib.pa_time_kernel(None, None, None) == B.PA_OK
    assert lib.pa_time_kernel(b"pa_token_attention", FAKE, FAKE) == B.PA_ERR_INVALID
    assert "no streaming kernel" in lib.pa_last_error().decode()
    assert lib.pa_time_kernel(b"pa_deslice", FAKE, None) == B.PA_ERR_INVALID
    assert lib.pa_time_kernel(b"pa_slice_aggregate_backward", FAKE, FAKE) == B.PA_OK
    assert lib.pa_time_kernel(None, None, None) == B.PA_OK


@fake_addresses
def test_stored_weights_argument_checks(lib):
    d = _dims()
    _, n = _ws_size(lib, d)
    assert lib.pa_deslice_w(ctypes.byref(d), None, FAKE, FAKE, FAKE, n, None) == B.PA_ERR_INVALID
    assert "W" in lib.pa_last_error().decode()
    assert lib.pa_deslice_backward_w(ctypes.byref(d), FAKE, None, FAKE, FAKE, n, None) == \
        B.PA_ERR_INVALID
    assert lib.pa_deslice_w(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, 16, None) == \
        B.PA_ERR_WORKSPACE
    sp = B.pa_slice_params(FAKE, None, None, 0.0)
    st = lib.pa_slice_aggregate_w(ctypes.byref(d), FAKE, None, ctypes.byref(sp), FAKE, FAKE,
                                  FAKE, None, FAKE, n, None)
    assert st == B.PA_ERR_INVALID and "W" in lib.pa_last_error().decode()



@fake_addresses
def test_heads_argument_checks(lib):
    far = FAKE + (1 << 32)
    # D not a multiple of 16 bytes' worth
    st = lib.pa_heads_relayout(100, 4, 6, B.PA_F32, 1, FAKE, far, None)
    assert st == B.PA_ERR_INVALID and "D" in lib.pa_last_error().decode()
    st = lib.pa_heads_relayout(100, 4, 4, B.PA_BF16, 1, FAKE, far, None)
    assert st == B.PA_ERR_INVALID
    # overlapping buffers, misaligned or missing pointers, empty shapes
    st = lib.pa_heads_relayout(100, 4, 8, B.PA_F32, 0, FAKE, FAKE + 64, None)
    assert st == B.PA_ERR_INVALID and "overlap" in lib.pa_last_error().decode()
    st = lib.pa_heads_relayout(100, 4, 8, B.PA_F32, 1, FAKE + 4, far, None)
    assert st == B.PA_ERR_INVALID and "aligned" in lib.pa_last_error().decode()
    st = lib.pa_heads_relayout(100, 4, 8, B.PA_F32, 1, None, far, None)
    assert st == B.PA_ERR_INVALID
    st = lib.pa_heads_relayout(0, 4, 8, B.PA_F32, 1, FAKE, far, None)
    assert st == B.PA_ERR_INVALID
    st = lib.pa_heads_relayout(100, 4, 8, 5, 1, FAKE, far, None)
    assert st == B.PA_ERR_INVALID
    # a block-diagonal matrix of more than 4096 rows; empty and misaligned
    st = lib.pa_heads_expand(64, 128, 1, FAKE, far, None)
    assert st == B.PA_ERR_INVALID
    st = lib.pa_heads_sum(0, 4, 0, FAKE, far, None)
    assert st == B.PA_ERR_INVALID
    st = lib.pa_heads_sum(2, 4, 0, FAKE + 2, far, None)
    assert st == B.PA_ERR_INVALID and "aligned" in lib.pa_last_error().decode()
    st = lib.pa_heads_expand(2, 4, 0, FAKE, None, None)
    assert st == B.PA_ERR_INVALID


@fake_addresses
def test_heads_batched_argument_checks(lib):
    d = _dims(N=1000, C=32, H=1, M=16, dtype=B.PA_BF16)
    far = FAKE + (1 << 32)
    hp = B.pa_heads_params(FAKE, None, None, None, 0)
    n = ctypes.c_size_t(0)
    assert lib.pa_heads_workspace_size(ctypes.byref(d), 4, ctypes.byref(n)) == B.PA_OK
    _, one = _ws_size(lib, d)
    assert n.value == 4 * one
    assert lib.pa_heads_workspace_size(ctypes.byref(d), 17, ctypes.byref(n)) == B.PA_ERR_INVALID
    # heads out of range, M not a multiple of 8, no params, workspace too small
    st = lib.pa_heads_slice_aggregate(ctypes.byref(d), 0, FAKE, None, ctypes.byref(hp), FAKE,
                                      FAKE, FAKE, far, n.value, None)
    assert st == B.PA_ERR_INVALID and "heads" in lib.pa_last_error().decode()
    d12 = _dims(N=1000, C=32, H=1, M=12, dtype=B.PA_BF16)
    st = lib.pa_heads_deslice(ctypes.byref(d12), 4, FAKE, None, ctypes.byref(hp), FAKE, FAKE,
                              far, n.value, None)
    assert st == B.PA_ERR_INVALID and "multiple of 8" in lib.pa_last_error().decode()
    st = lib.pa_heads_deslice_backward(ctypes.byref(d), 4, FAKE, None, None, FAKE, FAKE, far,
                                       n.value, None)
    assert st == B.PA_ERR_INVALID
    st = lib.pa_heads_slice_aggregate_backward(ctypes.byref(d), 4, FAKE, None, ctypes.byref(hp),
                                               None, None, None, None, None, FAKE, None, far,
                                               n.value - 256, None)
    assert st == B.PA_ERR_WORKSPACE
    # a misaligned b_t array
    hpn = B.pa_heads_params(FAKE, None, None, FAKE + 2, 0)
    st = lib.pa_heads_slice_aggregate(ctypes.byref(d), 4, FAKE, None, ctypes.byref(hpn), FAKE,
                                      FAKE, FAKE, far, n.value, None)
    assert st == B.PA_ERR_INVALID and "b_t" in lib.pa_last_error().decode()


def test_struct_layouts_match_header(tmp_path):
    """The ctypes structs of the binding have the sizes and field offsets the
    C compiler gives the header's structs."""
    import subprocess
    structs = {"pa_dims": B.pa_dims, "pa_slice_params": B.pa_slice_params,
               "pa_attn_params": B.pa_attn_params, "pa_slice_grads": B.pa_slice_grads,
               "pa_attn_grads": B.pa_attn_grads, "pa_heads_params": B.pa_heads_params}
    lines = ['#include <stdio.h>', '#include "pa.h"', "int main(void) {"]
    for name, cls in structs.items():
        lines.append(f'  printf("{name} sizeof %zu\\n", sizeof({name}));')
        for f in cls._fields_:
            lines.append(f'  printf("{name} {f[0]} %zu\\n", offsetof({name}, {f[0]}));')
    lines += ["  return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    subprocess.run(["gcc", "-std=c11", "-I", os.path.join(root, "include"), str(src), "-o",
                    str(exe)], check=True)
    got = {}
    for line in subprocess.run([str(exe)], check=True, capture_output=True,
                               text=True).stdout.splitlines():
        name, field, val = line.split()
        got[(name, field)] = int(val)
    for name, cls in structs.items():
        assert got[(name, "sizeof")] == ctypes.sizeof(cls), name
        for f in cls._fields_:
            assert got[(name, f[0])] == getattr(cls, f[0]).offset, (name, f[0])


@fake_addresses
def test_mlp_up_argument_checks(lib):
    F, K = 1024, 256
    # unserved K or F
    st = lib.pa_mlp_up(1000, 96, F, FAKE, FAKE, FAKE, FAKE, FAKE, 2 * F * K, None)
    assert st == B.PA_ERR_UNSUPPORTED
    st = lib.pa_mlp_up(1000, K, 1000, FAKE, FAKE, FAKE, FAKE, FAKE, 2 * F * K, None)
    assert st == B.PA_ERR_UNSUPPORTED
    # missing or misaligned pointers, small workspace, missing dY / W2
    st = lib.pa_mlp_up(1000, K, F, None, FAKE, FAKE, FAKE, FAKE, 2 * F * K, None)
    assert st == B.PA_ERR_INVALID and "X" in lib.pa_last_error().decode()
    st = lib.pa_mlp_up(1000, K, F, FAKE, FAKE + 4, FAKE, FAKE, FAKE, 2 * F * K, None)
    assert st == B.PA_ERR_INVALID and "W1" in lib.pa_last_error().decode()
    st = lib.pa_mlp_up(1000, K, F, FAKE, FAKE, FAKE, FAKE, FAKE, 2 * F * K - 1, None)
    assert st == B.PA_ERR_WORKSPACE
    st = lib.pa_mlp_up(0, K, F, FAKE, FAKE, FAKE, FAKE, FAKE, 2 * F * K, None)
    assert st == B.PA_ERR_INVALID
    st = lib.pa_mlp_up_backward(1000, K, F, FAKE, FAKE, FAKE, None, FAKE, FAKE, FAKE, 2 * F * K,
                                None)
    assert st == B.PA_ERR_INVALID and "dY" in lib.pa_last_error().decode()
    st = lib.pa_mlp_up_backward(1000, K, F, FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE, 2 * F * K,
                                None)
    assert st == B.PA_ERR_INVALID and "W2" in lib.pa_last_error().decode()


@fake_addresses
def test_stream_probe_argument_checks(lib):
    d = _dims(C=256, H=8, M=32, dtype=B.PA_BF16)
    # unknown or missing call names, missing tensors: host errors, nothing launched
    for call in (b"pa_token_attention", b"nope", None):
        st = lib.pa_stream_probe(ctypes.byref(d), call, FAKE, FAKE, None, FAKE, None)
        assert st == B.PA_ERR_INVALID
    st = lib.pa_stream_probe(ctypes.byref(d), b"pa_slice_aggregate_backward", FAKE, None, None,
                             FAKE, None)
    assert st == B.PA_ERR_INVALID  # dY required
    st = lib.pa_stream_probe(ctypes.byref(d), b"pa_deslice", FAKE, None, None, None, None)
    assert st == B.PA_ERR_INVALID  # out required
    st = lib.pa_stream_probe(ctypes.byref(_dims(C=48, H=4)), b"pa_deslice", FAKE + 8, None, None,
                             FAKE, None)
    assert st == B.PA_ERR_INVALID  # misaligned x
    assert lib.pa_last_error().decode() != ""


def test_heads_sum_batch_argument_checks(lib):
    # host validation only (nothing is launched): item counts outside [1, 8],
    # NULL items, an item that pa_heads_sum would reject
    items = (B.pa_heads_sum_item * 9)()
    assert lib.pa_heads_sum_batch(8, 0, items, None) == B.PA_ERR_INVALID
    assert lib.pa_heads_sum_batch(8, 9, items, None) == B.PA_ERR_INVALID
    assert lib.pa_heads_sum_batch(8, 1, None, None) == B.PA_ERR_INVALID
    items[0] = B.pa_heads_sum_item(None, None, 4, 0)  # NULL src and dst
    assert lib.pa_heads_sum_batch(8, 1, items, None) == B.PA_ERR_INVALID
    assert "pa_heads_sum_batch" in lib.pa_last_error().decode()

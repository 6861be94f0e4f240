"""Argument checks of the C ABI with real device buffers: each bad call is
refused with its status before anything is launched."""
import ctypes

import numpy as np
import pytest
import torch

import paper_2608_20725_amd as pkg

pytestmark = pytest.mark.gpu

EALIGN, EWORKSPACE, EOVERLAP, EBUFFER = -2, -6, -7, -8

N, Ci, H, W, Co, Kh, Kw, s = 2, 8, 10, 10, 16, 3, 3, 1


def _bufs(dtype=torch.float32):
    dev = "cuda"
    need = pkg.conv_workspace_bytes(N, Ci, H, W, Co, Kh, Kw, s, dtype)
    x = torch.zeros(N, H, W, Ci, dtype=dtype, device=dev)
    w = torch.zeros(Kh, Kw, Ci, Co, dtype=dtype, device=dev)
    ws = torch.zeros(need, dtype=torch.uint8, device=dev)
    out = torch.zeros(N, 8, 8, Co, dtype=dtype, device=dev)
    return x, w, ws, out, need


def _status(fn, *a):
    with pytest.raises(pkg.Im2winError) as e:
        fn(*a)
    return e.value.status


def test_workspace_too_small():
    x, w, ws, out, need = _bufs()
    assert _status(pkg.conv_im2win_transform, x, ws[:need - 16], Co, Kh, Kw, s) == EWORKSPACE
    assert _status(pkg.conv_im2win_fp32, ws[:need - 16], w, out, N, Ci, H, W, s) == EWORKSPACE


def test_misaligned_views():
    x, w, ws, out, need = _bufs()
    big = torch.zeros(need + 64, dtype=torch.uint8, device="cuda")
    assert _status(pkg.conv_im2win_transform, x, big[8:8 + need], Co, Kh, Kw, s) == EALIGN
    o = torch.zeros(out.numel() + 4, device="cuda")[1:1 + out.numel()].view(out.shape)
    assert _status(pkg.conv_im2win_fp32, ws, w, o, N, Ci, H, W, s) == EALIGN


def test_overlapping_buffers():
    x, w, ws, out, need = _bufs()
    flat = torch.zeros(need + out.numel() * 4, dtype=torch.uint8, device="cuda")
    wsv = flat[:need]
    o = flat[need - 256:need - 256 + out.numel() * 4].view(torch.float32).view(out.shape)
    assert _status(pkg.conv_im2win_fp32, wsv, w, o, N, Ci, H, W, s) == EOVERLAP


def test_host_pointer_refused():
    x, w, ws, out, need = _bufs()
    host = np.zeros(out.numel(), np.float32)
    lib = pkg.load_library()
    rc = lib.conv_im2win_fp32(ctypes.c_void_p(ws.data_ptr()), need, ctypes.c_void_p(w.data_ptr()),
                              ctypes.c_void_p(host.ctypes.data), N, Ci, H, W, Co, Kh, Kw, s, None)
    assert rc == EBUFFER


def test_buffer_smaller_than_layer():
    # an output allocation too small for the layer is refused, not overrun:
    # EBUFFER when the block ends before the output would, or EOVERLAP when
    # torch's caching allocator carved the block out of the segment that also
    # holds the workspace (the output range then runs into the workspace)
    x, w, ws, out, need = _bufs()
    lib = pkg.load_library()
    small = torch.cuda.caching_allocator_alloc(256)
    try:
        rc = lib.conv_im2win_fp32(ctypes.c_void_p(ws.data_ptr()), need,
                                  ctypes.c_void_p(w.data_ptr()), ctypes.c_void_p(small),
                                  64, Ci, H, W, Co, Kh, Kw, s, None)
        assert rc in (EBUFFER, EWORKSPACE, EOVERLAP)
    finally:
        torch.cuda.caching_allocator_delete(small)

"""The allocation-free mini-batch entry point (conv_im2win_chunked_noalloc),
called through the C ABI: its workspace is the library's static device
buffer.  Each call must give, bit for bit, what conv_im2win_chunked gives with
a caller-allocated workspace (same chunking, one stream), on two calls in a
row, the second with a smaller input (the buffer keeps the first call's
bytes); a request larger than the buffer is refused before anything runs."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import paper_2608_20725_amd as pkg
from gpu_util import TOL, oracle_inputs, rel_err, say
from paper_2608_20725_amd import workloads

pytestmark = pytest.mark.gpu

EWORKSPACE = -6
STATIC_BYTES = 128 << 20
DTYPES = [torch.float32, torch.float16, torch.bfloat16]
CODE = {torch.float32: 0, torch.float16: 1, torch.bfloat16: 2}


def _lib():
    lib = pkg.load_library()
    f = lib.conv_im2win_chunked_noalloc
    f.restype = ctypes.c_int
    f.argtypes = [ctypes.c_void_p] * 3 + [ctypes.c_int64] * 9 + [ctypes.c_int, ctypes.c_void_p]
    return f


def _inputs(shape, dtype, seed):
    N, Ci, H, W, Co, Kh, Kw, s = shape
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=seed)
    Ho, Wo = pkg.conv_output_dims(H, W, Kh, Kw, s)
    return x, w, x.to(dtype).contiguous().cuda(), w.to(dtype).contiguous().cuda(), (N, Ho, Wo, Co)


def _noalloc(f, xd, wd, shape, n_chunk, out_shape, dtype):
    N, Ci, H, W, Co, Kh, Kw, s = shape
    out = torch.full(out_shape, float("nan"), dtype=dtype, device="cuda")
    st = torch.cuda.current_stream().cuda_stream
    rc = f(xd.data_ptr(), wd.data_ptr(), out.data_ptr(), N, Ci, H, W, Co, Kh, Kw, s, n_chunk, CODE[dtype], st)
    return rc, out


def _with_workspace(xd, wd, shape, n_chunk, out_shape, dtype):
    N, Ci, H, W, Co, Kh, Kw, s = shape
    need = pkg.conv_chunked_workspace_bytes(N, Ci, H, W, Co, Kh, Kw, s, n_chunk, False, dtype)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    out = torch.full(out_shape, float("nan"), dtype=dtype, device="cuda")
    pkg.conv_im2win_chunked(xd, wd, out, ws, s, n_chunk)
    return out


@pytest.mark.parametrize("dtype", DTYPES, ids=["f32", "f16", "bf16"])
def test_noalloc_matches_chunked_twice(dtype):
    f = _lib()
    bits = torch.int32 if dtype == torch.float32 else torch.int16
    # second call smaller: fewer images, fewer channels, another kernel
    cases = [((12, 64, 30, 30, 96, 3, 3, 1), 5), ((3, 16, 14, 17, 24, 3, 3, 1), 2)]
    for k, (shape, n_chunk) in enumerate(cases):
        say("noalloc", dtype, shape, n_chunk)
        x, w, xd, wd, out_shape = _inputs(shape, dtype, seed=61 + k)
        rc, out = _noalloc(f, xd, wd, shape, n_chunk, out_shape, dtype)
        assert rc == 0, pkg.conv_im2win_strerror(rc)
        ref = _with_workspace(xd, wd, shape, n_chunk, out_shape, dtype)
        torch.cuda.synchronize()
        assert torch.equal(out.view(bits), ref.view(bits))
        xo, wo = oracle_inputs(x, w, dtype)
        o, a = oracle.conv(xo, wo, shape[7], with_abs=True)
        y = out.float().cpu().numpy().astype(np.float64)
        assert not np.isnan(y).any()
        assert rel_err(y, o, a) <= TOL[dtype]


def test_noalloc_refuses_more_than_the_buffer():
    f = _lib()
    # 56x56 C=64 fp32: a 64-image chunk needs ~149 MB of window tensor
    shape = (64, 64, 56, 56, 64, 3, 3, 1)
    N, Ci, H, W, Co, Kh, Kw, s = shape
    need = pkg.conv_chunked_workspace_bytes(N, Ci, H, W, Co, Kh, Kw, s, 64, False, torch.float32)
    assert need > STATIC_BYTES
    x, w, xd, wd, out_shape = _inputs(shape, torch.float32, seed=67)
    rc, out = _noalloc(f, xd, wd, shape, 64, out_shape, torch.float32)
    assert rc == EWORKSPACE
    torch.cuda.synchronize()
    assert torch.isnan(out).all()   # nothing ran
    # a chunking that fits runs
    rc, out = _noalloc(f, xd, wd, shape, 16, out_shape, torch.float32)
    assert rc == 0
    torch.cuda.synchronize()
    assert not torch.isnan(out).any()

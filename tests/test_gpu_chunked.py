"""Mini-batch im2win (conv_im2win_chunked): chunks of n_chunk images through a
one- or two-slot workspace, with and without a second stream.  The output must
equal the full-batch call bit for bit and match the oracle; the bytes after the
workspace must stay untouched."""
import numpy as np
import pytest
import torch

import paper_2608_20725_amd as pkg
from gpu_util import Run, check_full, say
from paper_2608_20725_amd import workloads

pytestmark = pytest.mark.gpu

DTYPES = [torch.float32, torch.float16, torch.bfloat16]
SHAPES = [
    (5, 16, 12, 12, 24, 3, 3, 1),     # row-per-pixel fp16 kernel
    (4, 64, 24, 24, 64, 3, 3, 1),     # column-staged fp16 kernel
    (3, 3, 20, 20, 16, 5, 5, 2),      # 3-channel stem: gather transform, unaligned windows
]
# (n_chunk, with a second stream)
CHUNKS = [(1, False), (2, True), (3, True), (4, False), (7, True)]
GUARD = 4096


def _run_chunked(x, w, s, dtype, n_chunk, two, aux=None):
    N, H, W, Ci = x.shape
    Kh, Kw, _, Co = w.shape
    Ho, Wo = pkg.conv_output_dims(H, W, Kh, Kw, s)
    need = pkg.conv_chunked_workspace_bytes(N, Ci, H, W, Co, Kh, Kw, s, n_chunk, two, dtype)
    ws_all = torch.full((need + GUARD,), 0xA5, dtype=torch.uint8, device="cuda")
    out = torch.full((N, Ho, Wo, Co), float("nan"), dtype=dtype, device="cuda")
    xd = x.to(dtype).contiguous().cuda()
    wd = w.to(dtype).contiguous().cuda()
    pkg.conv_im2win_chunked(xd, wd, out, ws_all[:need], s, n_chunk, aux_stream=aux)
    torch.cuda.synchronize()
    assert np.all(ws_all[need:].cpu().numpy() == 0xA5), "bytes written past the workspace"
    return out


@pytest.mark.parametrize("dtype", DTYPES, ids=["f32", "f16", "bf16"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda t: "x".join(map(str, t)))
def test_chunked_equals_full_batch(shape, dtype):
    N, Ci, H, W, Co, Kh, Kw, s = shape
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=23)
    full = Run(x, w, s, dtype)
    check_full(full, x, w)
    ref = full.out.cpu()
    aux = torch.cuda.Stream()
    for n_chunk, two in CHUNKS:
        say("chunked", shape, dtype, n_chunk, two)
        out = _run_chunked(x, w, s, dtype, n_chunk, two, aux if two else None)
        got = out.cpu()
        bits = torch.int32 if dtype == torch.float32 else torch.int16
        assert torch.equal(got.view(bits), ref.view(bits)), (n_chunk, two)


def test_chunked_back_to_back_reuses_workspace():
    """Two calls in a row on one workspace with a second stream: the second
    call's transforms must wait for the first call's convolutions."""
    shape = (6, 16, 14, 14, 32, 3, 3, 1)
    N, Ci, H, W, Co, Kh, Kw, s = shape
    x1, w1 = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=31)
    x2, w2 = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=32)
    dt = torch.float16
    ref1, ref2 = Run(x1, w1, s, dt).out.cpu(), Run(x2, w2, s, dt).out.cpu()
    need = pkg.conv_chunked_workspace_bytes(N, Ci, H, W, Co, Kh, Kw, s, 2, True, dt)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    Ho, Wo = pkg.conv_output_dims(H, W, Kh, Kw, s)
    o1 = torch.empty((N, Ho, Wo, Co), dtype=dt, device="cuda")
    o2 = torch.empty_like(o1)
    aux = torch.cuda.Stream()
    pkg.conv_im2win_chunked(x1.half().cuda(), w1.half().cuda(), o1, ws, s, 2, aux_stream=aux)
    pkg.conv_im2win_chunked(x2.half().cuda(), w2.half().cuda(), o2, ws, s, 2, aux_stream=aux)
    torch.cuda.synchronize()
    assert torch.equal(o1.cpu().view(torch.int16), ref1.view(torch.int16))
    assert torch.equal(o2.cpu().view(torch.int16), ref2.view(torch.int16))


def test_chunked_errors():
    shape = (4, 8, 10, 10, 16, 3, 3, 1)
    N, Ci, H, W, Co, Kh, Kw, s = shape
    x = torch.zeros(N, H, W, Ci, device="cuda")
    w = torch.zeros(Kh, Kw, Ci, Co, device="cuda")
    out = torch.zeros(N, 8, 8, Co, device="cuda")
    need = pkg.conv_chunked_workspace_bytes(N, Ci, H, W, Co, Kh, Kw, s, 2, True, torch.float32)
    ws = torch.zeros(need, dtype=torch.uint8, device="cuda")
    st = torch.cuda.Stream()                    # a created stream: non-NULL handle
    with pytest.raises(pkg.Im2winError) as e:   # the two streams must differ
        pkg.conv_im2win_chunked(x, w, out, ws, s, 2, stream=st, aux_stream=st)
    assert e.value.status == -1
    with pytest.raises(pkg.Im2winError) as e:   # two slots need more workspace than one
        pkg.conv_im2win_chunked(x, w, out, ws[:need - 256], s, 2, aux_stream=torch.cuda.Stream())
    assert e.value.status == -6
    with pytest.raises(pkg.Im2winError) as e:   # output overlapping the workspace
        pkg.conv_im2win_chunked(x, w, ws[:out.numel() * 4].view(torch.float32).view(out.shape), ws, s, 2)
    assert e.value.status == -7

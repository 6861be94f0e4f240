"""Mini-batch im2win (conv_im2win_chunked): chunks of n_chunk images through a
one- or two-slot workspace, with and without a second stream.  The output must
match the oracle, and equal the full-batch call bit for bit wherever both run
the same kernel; the bytes after the workspace must stay untouched.  At full
size: the benchmark's configuration (56x56 C=64, 128 images, 32-image chunks,
two streams) and chunkings whose smaller last chunk would select another
kernel (and packed-filter layout) on its own."""
import numpy as np
import pytest
import torch

import paper_2608_20725_amd as pkg
from gpu_util import Run, TOL, check_full, oracle_inputs, rel_err, sample_points, say
import oracle
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
    full_kernel = pkg.conv_im2win_kernel_name(N, Ci, H, W, Co, Kh, Kw, s, dtype)
    for n_chunk, two in CHUNKS:
        say("chunked", shape, dtype, n_chunk, two)
        out = _run_chunked(x, w, s, dtype, n_chunk, two, aux if two else None)
        check_out(out, x, w, s, dtype)
        chunk_kernel = pkg.conv_im2win_kernel_name(min(n_chunk, N), Ci, H, W, Co, Kh, Kw, s, dtype)
        if chunk_kernel == full_kernel:
            got = out.cpu()
            bits = torch.int32 if dtype == torch.float32 else torch.int16
            assert torch.equal(got.view(bits), ref.view(bits)), (n_chunk, two)


def check_out(out, x, w, s, dtype):
    """Every output of a small layer against the oracle."""
    xo, wo = oracle_inputs(x, w, dtype)
    ref, absref = oracle.conv(xo, wo, s, with_abs=True)
    y = out.float().cpu().numpy().astype(np.float64)
    assert not np.isnan(y).any(), "output element left unwritten"
    r = rel_err(y, ref, absref)
    assert r <= TOL[dtype], r


def check_out_sampled(out, x, w, s, dtype, images, seed):
    """All outputs of `images` plus 4096 random ones against the oracle,
    computed point by point on the images they touch."""
    N, Ho, Wo, Co = out.shape
    Kh, Kw, Ci, _ = w.shape
    pts = sample_points(N, Ho, Wo, Co, seed, full_images=images)
    imgs = np.unique(pts[:, 0])
    remap = {int(i): k for k, i in enumerate(imgs)}
    xo, wo = oracle_inputs(x[torch.from_numpy(imgs)], w, dtype)
    local = pts.copy()
    local[:, 0] = [remap[int(i)] for i in pts[:, 0]]
    ref, absref = oracle.conv_points(xo, wo, s, local)
    y = out.float().cpu().numpy()
    assert not np.isnan(y).any(), "output element left unwritten"
    got = y[pts[:, 0], pts[:, 1], pts[:, 2], pts[:, 3]].astype(np.float64)
    r = rel_err(got, ref, absref)
    assert r <= TOL[dtype], "max |err|/sum|x||w| = %.3g on %d sampled outputs" % (r, len(pts))
    return r, len(pts)


# (layer shape, n_chunk, dtype): the benchmark's mini-batch configuration in
# both precisions, and chunkings whose last chunk on its own would pick
# another kernel: 3x3 C=512 at 14x14 in 128-image chunks (a full chunk runs
# the column-staged 256 x 192 tile, the 32 images of the last chunk alone
# would run the row kernel, whose packed filter has another layout), and
# 56x56 C=64 fp32 in 100-image chunks (the 256-pixel tile; 28 images alone
# take the tap-split tile).
FULL_SIZE = [
    ((128, 64, 56, 56, 64, 3, 3, 1), 32, torch.float32),
    ((128, 64, 56, 56, 64, 3, 3, 1), 32, torch.float16),
    ((160, 512, 14, 14, 512, 3, 3, 1), 128, torch.float16),
    ((160, 512, 14, 14, 512, 3, 3, 1), 128, torch.bfloat16),
    ((128, 64, 56, 56, 64, 3, 3, 1), 100, torch.float32),
]


@pytest.mark.parametrize("case", FULL_SIZE, ids=lambda c: "x".join(map(str, c[0])) + "-c%d-%s" % (c[1], str(c[2])[6:]))
def test_chunked_full_size_against_oracle(case):
    shape, n_chunk, dtype = case
    N, Ci, H, W, Co, Kh, Kw, s = shape
    last = N - (N - 1) // n_chunk * n_chunk
    say("chunked full size", shape, n_chunk, dtype, "chunk kernel",
        pkg.conv_im2win_kernel_name(n_chunk, Ci, H, W, Co, Kh, Kw, s, dtype),
        "last chunk alone", pkg.conv_im2win_kernel_name(last, Ci, H, W, Co, Kh, Kw, s, dtype))
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=29)
    out = _run_chunked(x, w, s, dtype, n_chunk, True, torch.cuda.Stream())
    # images in the first chunk, across the first chunk boundary, and in the last chunk
    r, n = check_out_sampled(out, x, w, s, dtype, (0, n_chunk - 1, n_chunk, N - last, N - 1), seed=n_chunk)
    say("  max rel err %.3g over %d outputs" % (r, n))


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

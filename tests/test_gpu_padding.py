"""Zero padding folded into the transform, on the GPU against the oracle's
padded definitions: the padded window tensor bit for bit, and convolutions of
padded layers (the fp32 and fp16 kernels run unchanged on the padded extents)
to the usual bar."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import SENTINEL, TOL, WS_GUARD, oracle_inputs, rel_err, say
from paper_2608_20725_amd import workloads
import paper_2608_20725_amd as pkg

pytestmark = pytest.mark.gpu

DTYPES = [torch.float32, torch.float16]
DT_IDS = ["f32", "f16"]

# (N, C_i, H, W, K_h, K_w, s, pad_h, pad_w): vector (C_i*elt a multiple of 16
# bytes) and gather transforms, "same" padding, pads on one axis, pads larger
# than the filter, a filter that only fits thanks to the padding.
T_SHAPES = [
    (2, 8, 9, 7, 3, 3, 1, 1, 1), (1, 16, 6, 5, 3, 2, 2, 2, 1), (3, 4, 11, 13, 5, 3, 1, 2, 0),
    (2, 3, 12, 12, 3, 3, 1, 1, 1), (1, 5, 7, 9, 7, 2, 3, 3, 0), (2, 12, 4, 6, 1, 1, 2, 0, 2),
    (1, 64, 10, 9, 3, 3, 2, 1, 1), (1, 1, 3, 3, 5, 5, 1, 1, 1), (2, 3, 6, 6, 2, 2, 1, 4, 4),
]


def _id(t):
    return "x".join(map(str, t))


def _ws(nbytes):
    all_ = torch.full((nbytes + WS_GUARD,), SENTINEL, dtype=torch.uint8, device="cuda")
    return all_, all_[:nbytes]


@pytest.mark.parametrize("dtype", DTYPES, ids=DT_IDS)
@pytest.mark.parametrize("shape", T_SHAPES, ids=_id)
def test_padded_transform_bitwise(shape, dtype):
    N, Ci, H, W, Kh, Kw, s, ph, pw = shape
    say("padded transform", shape, dtype)
    x, _ = workloads.draw(N, Ci, H, W, 2, Kh, Kw, seed=sum(shape))
    xd = x.to(dtype).contiguous().cuda()
    need = pkg.conv_workspace_bytes(N, Ci, H + 2 * ph, W + 2 * pw, 2, Kh, Kw, s, dtype)
    ws_all, ws = _ws(need)
    pkg.conv_im2win_transform_padded(xd, ws, 2, Kh, Kw, s, ph, pw)
    torch.cuda.synchronize()
    ref = oracle.im2win_pad(x.to(dtype).numpy(), Kh, s, ph, pw)
    nb = ref.nbytes
    assert ws[:nb].cpu().numpy().tobytes() == ref.tobytes(), "padded window tensor differs"
    pad_end = (nb + 255) // 256 * 256 + 256
    assert np.all(ws[nb:pad_end].cpu().numpy() == 0), "pad not zeroed"
    assert np.all(ws_all[pad_end:].cpu().numpy() == SENTINEL), "transform wrote past the pad"


@pytest.mark.parametrize("dtype", DTYPES, ids=DT_IDS)
def test_pad_zero_is_the_plain_transform(dtype):
    N, Ci, H, W, Kh, Kw, s = 2, 8, 9, 10, 3, 3, 2
    x, _ = workloads.draw(N, Ci, H, W, 2, Kh, Kw, seed=3)
    xd = x.to(dtype).contiguous().cuda()
    need = pkg.conv_workspace_bytes(N, Ci, H, W, 2, Kh, Kw, s, dtype)
    _, a = _ws(need)
    _, b = _ws(need)
    pkg.conv_im2win_transform(xd, a, 2, Kh, Kw, s)
    pkg.conv_im2win_transform_padded(xd, b, 2, Kh, Kw, s, 0, 0)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def _padded_conv(x, w, s, ph, pw, dtype):
    N, H, W, Ci = x.shape
    Kh, Kw, _, Co = w.shape
    Hp, Wp = H + 2 * ph, W + 2 * pw
    Ho, Wo = pkg.conv_output_dims(Hp, Wp, Kh, Kw, s)
    xd = x.to(dtype).contiguous().cuda()
    wd = w.to(dtype).contiguous().cuda()
    _, ws = _ws(pkg.conv_workspace_bytes(N, Ci, Hp, Wp, Co, Kh, Kw, s, dtype))
    out = torch.full((N, Ho, Wo, Co), float("nan"), dtype=dtype, device="cuda")
    pkg.conv_im2win_transform_padded(xd, ws, Co, Kh, Kw, s, ph, pw)
    f = pkg.conv_im2win_fp32 if dtype == torch.float32 else pkg.conv_im2win_fp16
    f(ws, wd, out, N, Ci, Hp, Wp, s)
    torch.cuda.synchronize()
    return out.float().cpu().numpy().astype(np.float64)


# (N, C_i, H, W, C_o, K_h, K_w, s, pad_h, pad_w), one or more per kernel path:
# 16-byte-aligned windows (fp32 DMA-staged, fp16 column- and row-staged) and
# unaligned ones (fp32 4-byte granules, fp16 segment- and register-staged).
C_SHAPES = [
    (2, 16, 14, 14, 40, 3, 3, 1, 1, 1),     # "same" 3x3
    (1, 8, 9, 11, 24, 5, 5, 2, 2, 2),       # 5x5 stride 2
    (2, 64, 12, 12, 64, 7, 7, 1, 3, 3),     # "same" 7x7
    (2, 3, 30, 30, 20, 3, 3, 1, 1, 1),      # stem, "same"
    (1, 3, 40, 40, 96, 11, 11, 4, 2, 2),    # large-kernel stem with padding
    (1, 16, 5, 5, 8, 3, 3, 1, 4, 4),        # pad wider than the filter
    (1, 12, 30, 30, 48, 5, 4, 2, 1, 2),     # K_h != K_w, pad_h != pad_w
]


@pytest.mark.parametrize("dtype", DTYPES, ids=DT_IDS)
@pytest.mark.parametrize("shape", C_SHAPES, ids=_id)
def test_padded_conv(shape, dtype):
    N, Ci, H, W, Co, Kh, Kw, s, ph, pw = shape
    say("padded conv", shape, dtype)
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=31 + sum(shape))
    y = _padded_conv(x, w, s, ph, pw, dtype)
    xo, wo = oracle_inputs(x, w, dtype)
    ref, absref = oracle.conv_pad(xo, wo, s, ph, pw, with_abs=True)
    assert y.shape == ref.shape
    assert not np.isnan(y).any(), "output element left unwritten"
    r = rel_err(y, ref, absref)
    assert r <= TOL[dtype], "max |err|/sum|x||w| = %.3g" % r


@pytest.mark.parametrize("dtype", DTYPES, ids=DT_IDS)
@pytest.mark.parametrize("shape", C_SHAPES, ids=_id)
def test_padded_conv_integer_exact(shape, dtype):
    N, Ci, H, W, Co, Kh, Kw, s, ph, pw = shape
    say("padded conv int", shape, dtype)
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=37, dist="int2")
    y = _padded_conv(x, w, s, ph, pw, dtype)
    ref = oracle.conv_pad(x.double().numpy(), w.double().numpy(), s, ph, pw)
    if dtype == torch.float16:
        ref = ref.astype(np.float16).astype(np.float64)
    assert np.array_equal(y, ref)


@pytest.mark.parametrize("dtype", DTYPES, ids=DT_IDS)
def test_padded_resnet_layer(dtype):
    """A ResNet-style 3x3 "same" layer (56x56, 64 channels), 4 images, every
    output checked."""
    N, Ci, H, W, Co, K, s, p = 4, 64, 56, 56, 64, 3, 1, 1
    say("padded resnet layer", dtype)
    x, w = workloads.draw(N, Ci, H, W, Co, K, K, seed=41)
    y = _padded_conv(x, w, s, p, p, dtype)
    assert y.shape == (N, H, W, Co)
    xo, wo = oracle_inputs(x, w, dtype)
    ref, absref = oracle.conv_pad(xo, wo, s, p, p, with_abs=True)
    r = rel_err(y, ref, absref)
    assert r <= TOL[dtype], "max |err|/sum|x||w| = %.3g" % r

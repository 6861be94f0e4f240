"""im2win transform on the GPU against the oracle (Eq. 2): bit-exact, the pad
zeroed, nothing written past the workspace."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import Run, say
from oracle_checks import TINY
from paper_2608_20725_amd import workloads

pytestmark = pytest.mark.gpu

DTYPES = [torch.float32, torch.float16, torch.bfloat16]

# (N, C_i, H, W, K_h, K_w, s): vector path (C_i*elt multiple of 16 bytes),
# gather path (any other C_i), strips that are not a whole number of 16-byte
# granules, K_h = 1, K_h = H.
SHAPES = [t[:4] + t[5:] for t in [(N, Ci, H, W, Co, Kh, Kw, s) for (N, Ci, H, W, Co, Kh, Kw, s) in TINY]]
SHAPES += [
    (2, 8, 9, 7, 3, 2, 2), (1, 16, 6, 5, 2, 1, 1), (3, 4, 11, 13, 5, 3, 2),
    (2, 3, 12, 12, 3, 3, 1), (1, 5, 7, 9, 7, 2, 3), (2, 12, 10, 6, 1, 1, 2),
    (1, 64, 20, 18, 3, 3, 2), (1, 1, 5, 5, 5, 5, 1),
]


def _bits(t):
    """Host array of a tensor's element bits (numpy has no bfloat16; the
    transform only moves bits)."""
    return t.view(torch.int16).numpy() if t.dtype == torch.bfloat16 else t.numpy()


def _compare(run, x):
    xs = _bits(x.to(run.dtype))
    ref = oracle.im2win(xs, run.Kh, run.s)
    nb = run.window_bytes()
    got = run.ws[:nb].cpu().numpy()
    assert got.tobytes() == ref.tobytes(), "window tensor differs from Eq. 2"
    pad_end = (nb + 255) // 256 * 256 + 256
    assert np.all(run.ws[nb:pad_end].cpu().numpy() == 0), "pad not zeroed"
    rest = run.ws[pad_end:].cpu().numpy()
    assert np.all(rest == 0xA5), "transform wrote past the pad"
    run.check_workspace_guard()


@pytest.mark.parametrize("dtype", DTYPES, ids=["f32", "f16", "bf16"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_transform_small(shape, dtype):
    N, Ci, H, W, Kh, Kw, s = shape
    say("transform", shape, dtype)
    x, w = workloads.draw(N, Ci, H, W, 2, Kh, Kw, seed=sum(shape))
    run = Run(x, w, s, dtype, conv=False)
    _compare(run, x)


@pytest.mark.parametrize("dtype", DTYPES, ids=["f32", "f16", "bf16"])
@pytest.mark.parametrize("layer", workloads.CONFIGS, ids=lambda l: l.name)
def test_transform_configs_full(layer, dtype):
    """The four named configurations at full size, whole tensor compared."""
    say("transform", layer.name, dtype)
    x, w = workloads.draw_layer(layer)
    run = Run(x, w, layer.stride, dtype, conv=False)
    _compare(run, x)


@pytest.mark.parametrize("dtype", DTYPES, ids=["f32", "f16", "bf16"])
@pytest.mark.parametrize("layer", workloads.SWEEP, ids=lambda l: l.name)
def test_transform_sweep_sampled_strips(layer, dtype):
    """The sweep layers at full batch: the strips of images 0, N-1 and two
    random images compared bit for bit."""
    say("transform", layer.name, dtype)
    x, w = workloads.draw_layer(layer)
    run = Run(x, w, layer.stride, dtype, conv=False)
    rng = np.random.default_rng(layer.seed)
    imgs = sorted({0, layer.N - 1, *rng.integers(1, layer.N - 1, 2).tolist()})
    per_img = run.Ho * run.W * run.Kh * run.Ci * run.xd.element_size()
    for i in imgs:
        ref = oracle.im2win(_bits(x[i:i + 1].to(dtype)), run.Kh, run.s)
        got = run.ws[i * per_img:(i + 1) * per_img].cpu().numpy()
        assert got.tobytes() == ref.tobytes(), "image %d" % i
    nb = run.window_bytes()
    pad_end = (nb + 255) // 256 * 256 + 256
    assert np.all(run.ws[nb:pad_end].cpu().numpy() == 0), "pad not zeroed"
    run.check_workspace_guard()


@pytest.mark.parametrize("shape", [(4, 64, 30, 30, 3, 3, 1), (3, 8, 17, 19, 5, 3, 2)], ids=lambda s: "x".join(map(str, s)))
def test_transform_linear_block_order_same_bytes(shape, monkeypatch):
    """IM2WIN_TRANSFORM_ORDER=linear (the ablation of the XCD-aware block
    order) changes only which block copies which granules: same bytes."""
    N, Ci, H, W, Kh, Kw, s = shape
    x, w = workloads.draw(N, Ci, H, W, 2, Kh, Kw, seed=3)
    ref = Run(x, w, s, torch.float16, conv=False)
    monkeypatch.setenv("IM2WIN_TRANSFORM_ORDER", "linear")
    run = Run(x, w, s, torch.float16, conv=False)
    _compare(run, x)
    assert torch.equal(run.ws[:run.window_bytes()], ref.ws[:ref.window_bytes()])


# Unaligned windows (C_i * elt not a multiple of 16 bytes) take the element
# gather: odd channel counts, strips that end inside a granule, K_h = H, a
# tall filter over a wide input, stride > K.
# The 3-channel layers' one-load-per-pixel gather (fp32; fp16 and bf16 with
# K_h <= 3) against the element gather: the same bytes, pad included, on odd
# and even widths, strides up to the filter height, and the Table I stems.
PIECES3 = [(2, 3, 12, 13, 3, 3, 1), (2, 3, 10, 11, 2, 2, 2), (1, 3, 7, 6, 1, 1, 1), (3, 3, 17, 16, 5, 5, 2),
           (1, 3, 23, 31, 7, 7, 3), (2, 3, 29, 27, 11, 11, 4), (1, 3, 11, 9, 11, 3, 1), (2, 3, 9, 40, 3, 3, 3),
           (2, 3, 227, 227, 11, 11, 4), (2, 3, 227, 227, 7, 7, 2), (2, 3, 224, 224, 3, 3, 1)]


@pytest.mark.parametrize("dtype", DTYPES, ids=["f32", "f16", "bf16"])
@pytest.mark.parametrize("shape", PIECES3, ids=lambda s: "x".join(map(str, s)))
def test_transform_3ch_pieces_equal_gather(shape, dtype, monkeypatch):
    N, Ci, H, W, Kh, Kw, s = shape
    x, w = workloads.draw(N, Ci, H, W, 2, Kh, Kw, seed=7 + sum(shape))
    outs = []
    for kernel in ("pieces", "gather"):
        monkeypatch.setenv("IM2WIN_TRANSFORM_KERNEL", kernel)
        say("transform", kernel, shape, dtype)
        run = Run(x, w, s, dtype, conv=False)
        if not outs:
            _compare(run, x)
        outs.append(run.ws.cpu())
    assert torch.equal(outs[0], outs[1])


UNALIGNED = [(2, 3, 12, 12, 3, 3, 1), (3, 5, 11, 13, 5, 3, 2), (1, 7, 9, 31, 9, 2, 3), (2, 1, 8, 8, 8, 8, 1),
             (2, 3, 227, 40, 11, 11, 4), (1, 3, 30, 300, 27, 5, 1), (2, 6, 10, 10, 2, 2, 3)]


@pytest.mark.parametrize("dtype", DTYPES, ids=["f32", "f16", "bf16"])
@pytest.mark.parametrize("shape", UNALIGNED, ids=lambda s: "x".join(map(str, s)))
def test_transform_unaligned(shape, dtype):
    N, Ci, H, W, Kh, Kw, s = shape
    say("unaligned transform", shape, dtype)
    x, w = workloads.draw(N, Ci, H, W, 2, Kh, Kw, seed=5 + sum(shape))
    run = Run(x, w, s, dtype, conv=False)
    _compare(run, x)

"""Filter dilation (an extension of the paper's convolution) on the GPU:
conv_im2win_transform_dilated against the oracle's dilated window tensor bit
for bit, conv_im2win_dilated against the oracle's dilated convolution (fp32,
fp16, bf16; tolerances as for the undilated calls), integer inputs exactly,
every kernel family and variant the dilated layout reaches, and dilation 1
reproducing the undilated calls bit for bit."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_20725_amd as pkg
from gpu_util import GUARD, SENTINEL, TOL, WS_GUARD, oracle_inputs, rel_err, say, assert_kernel
from paper_2608_20725_amd import workloads

pytestmark = pytest.mark.gpu

DTYPES = [torch.float32, torch.float16, torch.bfloat16]
DT_IDS = ["f32", "f16", "bf16"]

# N, C_i, H, W, C_o, K_h, K_w, s, pad_h, pad_w, d
SHAPES = [
    (2, 8, 17, 19, 24, 3, 3, 1, 2, 2, 2),      # "same" 3x3, d = 2
    (1, 16, 21, 23, 40, 3, 2, 2, 1, 3, 3),     # K_h != K_w, stride 2, d = 3, pad_h != pad_w
    (2, 3, 20, 20, 16, 3, 3, 1, 0, 0, 4),      # 3 channels: unaligned windows, d = 4
    (1, 64, 30, 30, 130, 3, 3, 1, 2, 2, 2),    # C_o ragged past 128
    (3, 12, 15, 31, 33, 5, 5, 3, 4, 4, 2),     # stride 3 > d, padded width not a multiple of d
    (1, 32, 9, 40, 64, 1, 1, 1, 0, 0, 3),      # 1x1: dilation changes nothing
    (2, 4, 13, 13, 8, 2, 2, 1, 0, 0, 12),      # dilated filter as large as the input
    (2, 20, 12, 45, 72, 3, 3, 1, 1, 1, 5),     # C_i = 20: 8-byte aligned windows, d = 5
]


def _id(t):
    return "x".join(map(str, t))


def _bits(t):
    return t.view(torch.int16).numpy() if t.dtype == torch.bfloat16 else t.numpy()


class DilRun:
    """Dilated transform (+ conv) through the C ABI with guard bands."""

    def __init__(self, x, w, s, ph, pw, d, dtype, conv=True):
        dev = torch.device("cuda")
        self.N, self.H, self.W, self.Ci = x.shape
        self.Kh, self.Kw, _, self.Co = w.shape
        self.s, self.ph, self.pw, self.d, self.dtype = s, ph, pw, d, dtype
        self.Hp, self.Wp = self.H + 2 * ph, self.W + 2 * pw
        self.Ho, self.Wo = pkg.conv_output_dims_dilated(self.Hp, self.Wp, self.Kh, self.Kw, s, d)
        self.need = pkg.conv_workspace_bytes_dilated(self.N, self.Ci, self.Hp, self.Wp, self.Co, self.Kh, self.Kw,
                                                     s, d, dtype)
        self.xd = x.to(dtype).contiguous().to(dev)
        self.wd = w.to(dtype).contiguous().to(dev)
        self.ws_all = torch.full((self.need + WS_GUARD,), SENTINEL, dtype=torch.uint8, device=dev)
        self.ws = self.ws_all[:self.need]
        n_out = self.N * self.Ho * self.Wo * self.Co
        self.out_all = torch.full((GUARD + n_out + GUARD,), float("nan"), dtype=dtype, device=dev)
        self.out = self.out_all[GUARD:GUARD + n_out].view(self.N, self.Ho, self.Wo, self.Co)
        pkg.conv_im2win_transform_dilated(self.xd, self.ws, self.Co, self.Kh, self.Kw, s, ph, pw, d)
        if conv:
            pkg.conv_im2win_dilated(self.ws, self.wd, self.out, self.N, self.Ci, self.Hp, self.Wp, s, d)
        torch.cuda.synchronize()

    def check_guards(self):
        assert np.all(self.ws_all[self.need:].cpu().numpy() == SENTINEL), "bytes written past the workspace"
        g = self.out_all.cpu()
        assert torch.isnan(g[:GUARD].float()).all() and torch.isnan(g[-GUARD:].float()).all(), \
            "write outside the output"

    def out_np(self):
        return self.out.float().cpu().numpy().astype(np.float64)


def _check_conv(run, x, w):
    xo, wo = oracle_inputs(x, w, run.dtype)
    ref, absref = oracle.conv_dil(xo, wo, run.s, run.ph, run.pw, run.d, with_abs=True)
    y = run.out_np()
    assert y.shape == ref.shape
    assert not np.isnan(y).any(), "output element left unwritten"
    r = rel_err(y, ref, absref)
    assert r <= TOL[run.dtype], "max |err|/sum|x||w| = %.3g" % r
    return r


@pytest.mark.parametrize("dtype", DTYPES, ids=DT_IDS)
@pytest.mark.parametrize("shape", SHAPES, ids=_id)
def test_dilated_transform_bitwise(shape, dtype):
    N, Ci, H, W, Co, Kh, Kw, s, ph, pw, d = shape
    say("dilated transform", shape, dtype)
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=sum(shape))
    run = DilRun(x, w, s, ph, pw, d, dtype, conv=False)
    ref = oracle.im2win_dil(_bits(x.to(dtype)), Kh, s, ph, pw, d)
    nb = ref.nbytes
    assert run.ws[:nb].cpu().numpy().tobytes() == ref.tobytes(), "dilated window tensor differs"
    pad_end = (nb + 255) // 256 * 256 + 256
    assert np.all(run.ws[nb:pad_end].cpu().numpy() == 0), "pad not zeroed"
    assert np.all(run.ws[pad_end:].cpu().numpy() == SENTINEL), "transform wrote past the pad"
    run.check_guards()


@pytest.mark.parametrize("dtype", DTYPES, ids=DT_IDS)
@pytest.mark.parametrize("shape", SHAPES, ids=_id)
def test_dilated_conv(shape, dtype):
    N, Ci, H, W, Co, Kh, Kw, s, ph, pw, d = shape
    say("dilated conv", shape, dtype)
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=3 + sum(shape))
    run = DilRun(x, w, s, ph, pw, d, dtype)
    _check_conv(run, x, w)
    run.check_guards()


@pytest.mark.parametrize("dtype", DTYPES, ids=DT_IDS)
@pytest.mark.parametrize("shape", SHAPES, ids=_id)
def test_dilated_conv_integer_exact(shape, dtype):
    N, Ci, H, W, Co, Kh, Kw, s, ph, pw, d = shape
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=29, dist="int2")
    run = DilRun(x, w, s, ph, pw, d, dtype)
    ref = oracle.conv_dil(x.double().numpy(), w.double().numpy(), s, ph, pw, d)
    if dtype != torch.float32:   # the one rounding on store
        ref = torch.from_numpy(ref).to(dtype).double().numpy()
    assert np.array_equal(run.out_np(), ref)


@pytest.mark.parametrize("dtype", DTYPES, ids=DT_IDS)
@pytest.mark.parametrize("shape", [(2, 8, 11, 13, 20, 3, 3, 1, 1, 1), (1, 3, 12, 17, 16, 3, 2, 2, 2, 0),
                                   (1, 16, 9, 9, 130, 2, 3, 1, 0, 1)], ids=_id)
def test_dilation_one_is_the_undilated_path(shape, dtype):
    """Dilation 1: the same window tensor as the padded transform and the same
    output bits as the plain conv entry points."""
    N, Ci, H, W, Co, Kh, Kw, s, ph, pw = shape
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=41)
    run = DilRun(x, w, s, ph, pw, 1, dtype)
    ws2 = torch.empty_like(run.ws)
    pkg.conv_im2win_transform_padded(run.xd, ws2, Co, Kh, Kw, s, ph, pw)
    out2 = torch.empty_like(run.out)
    pkg.conv_for_dtype(dtype)(ws2, run.wd, out2, N, Ci, run.Hp, run.Wp, s)
    torch.cuda.synchronize()
    nb = N * run.Ho * run.Wp * Kh * Ci * run.xd.element_size()
    assert torch.equal(run.ws[:nb], ws2[:nb])
    bits = torch.int32 if dtype == torch.float32 else torch.int16
    assert torch.equal(run.out.view(bits), out2.view(bits))


# Every kernel variant the dilated layout reaches, forced through the tuning
# variables (the column- and segment-staged fp16 kernels step aside for
# dilated layers; the register-staged ones and every row-per-pixel tile and
# fp32 variant compute window starts through the dilated rule).
VARIANTS = [
    ("IM2WIN_FP32_KERNEL", ["p8c8l8s2k16", "p6c8l8s2k16", "p4c8l8s2k16", "p4c16l1s2k16", "p8c8l8s2k16t4",
                            "p4c8l8s2k16t4", "regs"],
     (2, 16, 14, 17, 72, 3, 3, 1, 2, 2, 2), torch.float32),
    ("IM2WIN_FP32_KERNEL", ["p8c8l8s2k16g4", "p6c8l8s2k16g4", "p4c8l8s2k16g4", "p4c12l8s2k16g4", "regs"],
     (2, 3, 20, 20, 16, 3, 3, 1, 0, 0, 4),
     torch.float32),
    ("IM2WIN_FP32_KERNEL", ["p4c12l8s2k16", "p8c12l8s2k16"], (2, 16, 14, 17, 96, 3, 3, 1, 2, 2, 2), torch.float32),
    ("IM2WIN_FP16_TILE", ["c32p128s3", "c64p128s3", "c128p128s2", "c256p256s2w8", "c128p256s2w8", "c128p128s1"],
     (2, 16, 14, 17, 72, 3, 3, 1, 2, 2, 2), torch.float16),
    ("IM2WIN_FP16_KERNEL", ["regs"], (2, 16, 14, 17, 72, 3, 3, 1, 2, 2, 2), torch.float16),
    ("IM2WIN_FP16_KERNEL", ["regs"], (2, 3, 20, 20, 16, 3, 3, 1, 0, 0, 4), torch.bfloat16),
]


@pytest.mark.parametrize("case", VARIANTS, ids=lambda c: c[0] + "-" + _id(c[2]) + "-" + str(c[3])[6:])
def test_dilated_kernel_variants(case, monkeypatch):
    var, names, shape, dtype = case
    N, Ci, H, W, Co, Kh, Kw, s, ph, pw, d = shape
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=43)
    for name in names:
        say("dilated variant", var, name, shape)
        monkeypatch.setenv(var, name)
        if var == "IM2WIN_FP16_TILE":
            monkeypatch.setenv("IM2WIN_FP16_KERNEL", "pipe")
        assert_kernel((N, Ci, H + 2 * ph, W + 2 * pw, Co, Kh, Kw, s), dtype, var, name, dilation=d)
        run = DilRun(x, w, s, ph, pw, d, dtype)
        _check_conv(run, x, w)
        run.check_guards()


@pytest.mark.parametrize("dtype", DTYPES, ids=DT_IDS)
def test_dilated_atrous_layer(dtype):
    """An atrous (DeepLab-style) layer: 3x3, d = 2, 'same' padding, 256
    channels at 33x33, batch 8; every output against the oracle."""
    N, Ci, H, W, Co, K, s, pad, d = 8, 256, 33, 33, 256, 3, 1, 2, 2
    x, w = workloads.draw(N, Ci, H, W, Co, K, K, seed=47)
    run = DilRun(x, w, s, pad, pad, d, dtype)
    assert (run.Ho, run.Wo) == (H, W)
    y = run.out.float().cpu().numpy()
    assert not np.isnan(y).any()
    xo, wo = oracle_inputs(x, w, dtype)
    ref, absref = oracle.conv_dil(xo, wo, s, pad, pad, d, with_abs=True)
    r = rel_err(y.astype(np.float64), ref, absref)
    say("  atrous layer max rel err %.3g" % r)
    assert r <= TOL[dtype]
    run.check_guards()

"""K split of the row-per-pixel fp16 kernel (IM2WIN_FP16_SPLIT): ks blocks
per output tile each sum one range of 64-tap stages, and a second kernel adds
the ks fp32 partial tiles in a fixed order.  Checked against the fp64 oracle
at the 16-bit bars, run-to-run bit equality (the order of the final additions
does not depend on which block finishes first), and the workspace the split
needs beyond the default plan's."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_20725_amd as pkg
from gpu_util import TOL, check_full, oracle_inputs, rel_err, say

pytestmark = pytest.mark.gpu

EWORKSPACE = -6

# (N, C_i, H, W, C_o, K_h, K_w, s): ragged pixel tiles, C_o not a multiple of
# 128, taps past K in the last stage, one tile only, many tiles per image
SHAPES = [
    (2, 64, 9, 9, 128, 3, 3, 1),       # K = 576: 9 stages
    (3, 40, 11, 13, 200, 3, 3, 1),     # K = 360 (ragged stage), C_o ragged
    (1, 512, 7, 7, 512, 3, 3, 1),      # the 3x3 512-channel 7x7 layer, one image
    (2, 96, 12, 12, 130, 5, 5, 1),     # K = 2400
    (1, 256, 4, 4, 64, 1, 1, 1),       # one 128 x 128 tile, 4 stages
]


def split_bytes(N, Ci, H, W, Co, Kh, Kw, s, ks):
    Ho, Wo = pkg.conv_output_dims(H, W, Kh, Kw, s)
    P = N * Ho * Wo
    tiles = -(-P // 128) * -(-Co // 128)
    return ks * tiles * 128 * 128 * 4


def run_split(x, w, s, dtype, ks, monkeypatch, extra=True):
    N, H, W, Ci = x.shape
    Kh, Kw, _, Co = w.shape
    monkeypatch.setenv("IM2WIN_FP16_TILE", "c128p128s2")
    monkeypatch.setenv("IM2WIN_FP16_SPLIT", str(ks))
    name = pkg.conv_im2win_kernel_name(N, Ci, H, W, Co, Kh, Kw, s, dtype)
    assert name == "conv_fp16_pipe c128p128s2" + (" k%d" % ks if ks > 1 else ""), name
    need = pkg.conv_workspace_bytes(N, Ci, H, W, Co, Kh, Kw, s, dtype)
    if extra:
        need += split_bytes(N, Ci, H, W, Co, Kh, Kw, s, ks)
    dev = torch.device("cuda")
    ws = torch.full((need,), 0xA5, dtype=torch.uint8, device=dev)
    xd, wd = x.to(dtype).contiguous().to(dev), w.to(dtype).contiguous().to(dev)
    Ho, Wo = pkg.conv_output_dims(H, W, Kh, Kw, s)
    out = torch.full((N, Ho, Wo, Co), float("nan"), dtype=dtype, device=dev)
    pkg.conv_im2win_transform(xd, ws, Co, Kh, Kw, s)
    pkg.conv_for_dtype(dtype)(ws, wd, out, N, Ci, H, W, s)
    torch.cuda.synchronize()
    return out, ws, wd


def _id(t):
    return "x".join(map(str, t))


@pytest.mark.parametrize("dtype", [torch.float16, torch.bfloat16], ids=["f16", "bf16"])
@pytest.mark.parametrize("shape", SHAPES, ids=_id)
def test_split_against_oracle_and_reproducible(shape, dtype, monkeypatch):
    N, Ci, H, W, Co, Kh, Kw, s = shape
    g = torch.Generator().manual_seed(7)
    x = torch.rand((N, H, W, Ci), generator=g) * 2 - 1
    w = torch.rand((Kh, Kw, Ci, Co), generator=g) * 2 - 1
    xo, wo = oracle_inputs(x, w, dtype)
    ref, absref = oracle.conv(xo, wo, s, with_abs=True)
    nst = -(-(Kh * Kw * Ci) // 64)
    for ks in (2, 3, 4):
        if (ks - 1) * -(-nst // ks) >= nst:
            continue   # an empty K range: the planner refuses it (CPU test)
        say("split", _id(shape), dtype, ks)
        out, ws, wd = run_split(x, w, s, dtype, ks, monkeypatch)
        y = out.float().cpu().numpy().astype(np.float64)
        assert not np.isnan(y).any(), "output element left unwritten"
        r = rel_err(y, ref, absref)
        assert r <= TOL[dtype], "ks=%d: max |err|/sum|x||w| = %.3g" % (ks, r)
        first = out.clone()
        for _ in range(3):
            pkg.conv_for_dtype(dtype)(ws, wd, out, N, Ci, H, W, s)
            torch.cuda.synchronize()
            assert torch.equal(first.view(torch.int16), out.view(torch.int16)), "ks=%d not reproducible" % ks


def test_split_integer_inputs_exact(monkeypatch):
    # small integers: every partial sum and the total are exact in fp32, so the
    # split sums the same value as the oracle, before one rounding to fp16
    N, Ci, H, W, Co, Kh, Kw, s = (2, 64, 9, 9, 128, 3, 3, 1)
    g = torch.Generator().manual_seed(3)
    x = torch.randint(-2, 3, (N, H, W, Ci), generator=g).float()
    w = torch.randint(-2, 3, (Kh, Kw, Ci, Co), generator=g).float()
    ref = oracle.conv(x.double().numpy(), w.double().numpy(), s)
    want = torch.from_numpy(ref).half().float().numpy()
    for ks in (2, 3):   # 9 stages: 2 ranges of 5 and 4, 3 of 3
        out, _, _ = run_split(x, w, s, torch.float16, ks, monkeypatch)
        assert np.array_equal(out.float().cpu().numpy(), want)


def test_split_needs_its_workspace(monkeypatch):
    # the default plan of this layer is unsplit: its workspace is too small
    # for a forced split, which the call refuses before launching anything
    x = torch.rand((2, 9, 9, 64)) * 2 - 1
    w = torch.rand((3, 3, 64, 128)) * 2 - 1
    with pytest.raises(pkg.Im2winError) as e:
        run_split(x, w, 1, torch.float16, 2, monkeypatch, extra=False)
    assert e.value.status == EWORKSPACE

"""The short-window kernels for windows that are not 16-byte aligned (the
3-channel stems): fp16/bf16 on the matrix cores (at most 160 taps) and fp32
on the vector ALUs (at most 32 taps).  fp16: every output against the fp64
oracle, the
same bits as the segment-staged kernel where both run (both add the 16-tap
k-steps of each window in order on the same matrix instruction), ragged last
blocks and tiles over many images, and non-finite inputs kept in their own
windows (taps past K are cleared before the multiply)."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import Run, TOL, assert_kernel, check_full, oracle_inputs, rel_err, say
from paper_2608_20725_amd import workloads

pytestmark = pytest.mark.gpu

# (N, C_i, H, W, C_o, K_h, K_w, s)
SHAPES = [
    (2, 3, 30, 31, 64, 3, 3, 1),     # 27 taps, 1682 pixels: a ragged last block
    (3, 1, 17, 40, 8, 3, 3, 1),      # C_i = 1, C_o = 8: one 16-byte chunk per row
    (1, 3, 32, 32, 16, 3, 3, 1),     # the tiny layer
    (2, 5, 19, 23, 40, 3, 3, 2),     # C_i = 5, stride 2, C_o = 40 (5 of 8 row chunks)
    (2, 3, 40, 37, 96, 4, 4, 1),     # 48 taps, three channel blocks
    (2, 3, 25, 27, 128, 5, 5, 1),    # 75 taps (forced), four channel blocks
    (2, 3, 41, 45, 64, 7, 7, 2),     # 147 taps (forced), ten k-steps
    (40, 3, 5, 5, 24, 5, 5, 1),      # one output pixel per image: blocks span 32 images
    (300, 3, 4, 4, 16, 2, 2, 1),     # many tiny images
]


def _id(t):
    return "x".join(map(str, t))


@pytest.mark.parametrize("dtype", [torch.float16, torch.bfloat16], ids=["f16", "bf16"])
@pytest.mark.parametrize("shape", SHAPES, ids=_id)
def test_stem_against_oracle_and_segment_kernel(shape, dtype, monkeypatch):
    N, Ci, H, W, Co, Kh, Kw, s = shape
    say("stem", shape, dtype)
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=31)
    monkeypatch.setenv("IM2WIN_FP16_KERNEL", "stem")
    assert_kernel(shape, "f16" if dtype == torch.float16 else "bf16", "IM2WIN_FP16_KERNEL", "stem")
    run = Run(x, w, s, dtype)
    check_full(run, x, w)
    run.check_out_guards()
    run.check_workspace_guard()
    mine = run.out.clone()
    monkeypatch.delenv("IM2WIN_FP16_KERNEL")
    monkeypatch.setenv("IM2WIN_FP16_SEG", "s64p256")
    try:
        other = Run(x, w, s, dtype)
    except Exception as e:   # the segment kernel does not fit every shape here
        if "invalid argument" in str(e):
            return
        raise
    assert torch.equal(mine.view(torch.int16), other.out.view(torch.int16))


# An output of 128 MiB or more leaves through streamed (nontemporal) buffer
# stores: every output against the oracle, the guard bytes after it, and the
# same bits as the segment-staged kernel's cached stores; 1,172,184 pixels,
# so the last 32-pixel block is ragged.
def test_stem_streamed_output(monkeypatch):
    shape = (24, 3, 223, 223, 64, 3, 3, 1)
    N, Ci, H, W, Co, Kh, Kw, s = shape
    assert N * (H - Kh + 1) * (W - Kw + 1) * Co * 2 >= 128 << 20
    say("stem streamed", shape)
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=37)
    assert_kernel(shape, "f16", "IM2WIN_FP16_KERNEL", "stem")
    run = Run(x, w, s, torch.float16)
    check_full(run, x, w)
    run.check_out_guards()
    mine = run.out.clone()
    monkeypatch.setenv("IM2WIN_FP16_SEG", "s64p256")
    other = Run(x, w, s, torch.float16)
    assert torch.equal(mine.view(torch.int16), other.out.view(torch.int16))


@pytest.mark.parametrize("shape", [(2, 3, 12, 40, 64, 3, 3, 1), (2, 3, 15, 33, 32, 5, 5, 2)], ids=_id)
def test_stem_nonfinite_inputs_stay_in_their_windows(shape, monkeypatch):
    N, Ci, H, W, Co, Kh, Kw, s = shape
    monkeypatch.setenv("IM2WIN_FP16_KERNEL", "stem")
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=29)
    rng = np.random.default_rng(29)
    for v in (float("inf"), float("-inf"), float("nan"), float("inf")):
        x[rng.integers(N), rng.integers(H), rng.integers(W), rng.integers(Ci)] = v
    run = Run(x, w, s, torch.float16)
    xo, wo = oracle_inputs(x, w, torch.float16)
    with np.errstate(invalid="ignore", over="ignore"):
        ref, absref = oracle.conv(xo, wo, s, with_abs=True)
    y = run.out_np()
    fin = np.isfinite(ref)
    assert (~fin).any() and fin.any()
    assert np.array_equal(np.isfinite(y), fin), "%d outputs differ in finiteness" % int(
        (np.isfinite(y) != fin).sum())
    r = rel_err(y[fin], ref[fin], absref[fin])
    assert r <= TOL[torch.float16], "max |err|/sum|x||w| = %.3g" % r


def test_stem_integer_inputs_exact(monkeypatch):
    N, Ci, H, W, Co, Kh, Kw, s = (3, 3, 20, 27, 64, 3, 3, 1)
    monkeypatch.setenv("IM2WIN_FP16_KERNEL", "stem")
    g = torch.Generator().manual_seed(5)
    x = torch.randint(-3, 4, (N, H, W, Ci), generator=g).float()
    w = torch.randint(-3, 4, (Kh, Kw, Ci, Co), generator=g).float()
    run = Run(x, w, s, torch.float16)
    ref = oracle.conv(x.double().numpy(), w.double().numpy(), s)
    assert np.array_equal(run.out.float().cpu().numpy(), torch.from_numpy(ref).half().float().numpy())


# fp32: up to 32 taps
SHAPES32 = [s for s in SHAPES if s[5] * s[6] * s[1] <= 32 and s[4] % 4 == 0] + [
    (2, 5, 19, 23, 36, 2, 3, 1),     # 30 taps, C_o = 36: a ragged 32-channel pass
    (3, 3, 21, 50, 100, 3, 3, 2),    # C_o = 100: four passes, the last with one chunk
]


@pytest.mark.parametrize("shape", SHAPES32, ids=_id)
def test_stem32_against_oracle_and_dma_kernel(shape, monkeypatch):
    N, Ci, H, W, Co, Kh, Kw, s = shape
    say("stem32", shape)
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=37)
    monkeypatch.setenv("IM2WIN_FP32_KERNEL", "stem")
    assert_kernel(shape, "f32", "IM2WIN_FP32_KERNEL", "stem")
    run = Run(x, w, s, torch.float32)
    check_full(run, x, w)
    run.check_out_guards()
    run.check_workspace_guard()
    # the DMA-staged kernel adds the same taps in the same order
    monkeypatch.setenv("IM2WIN_FP32_KERNEL", "p6c8l8s2k16g4")
    other = Run(x, w, s, torch.float32)
    assert torch.equal(run.out.view(torch.int32), other.out.view(torch.int32))


def test_stem32_nonfinite_and_integer(monkeypatch):
    monkeypatch.setenv("IM2WIN_FP32_KERNEL", "stem")
    N, Ci, H, W, Co, Kh, Kw, s = (2, 3, 14, 40, 64, 3, 3, 1)
    g = torch.Generator().manual_seed(8)
    x = torch.randint(-4, 5, (N, H, W, Ci), generator=g).float()
    w = torch.randint(-4, 5, (Kh, Kw, Ci, Co), generator=g).float()
    run = Run(x, w, s, torch.float32)
    ref = oracle.conv(x.double().numpy(), w.double().numpy(), s)
    assert np.array_equal(run.out.cpu().numpy(), ref.astype(np.float32))
    x[1, 5, 7, 2] = float("inf")
    x[0, 0, 39, 0] = float("nan")
    run = Run(x, w, s, torch.float32)
    with np.errstate(invalid="ignore", over="ignore"):
        ref = oracle.conv(x.double().numpy(), w.double().numpy(), s)
    assert np.array_equal(np.isfinite(run.out.cpu().numpy()), np.isfinite(ref))

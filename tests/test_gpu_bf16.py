"""bf16 windowed convolution (matrix cores, fp32 accumulation, bf16 output)
on the GPU against the fp64 oracle computed on the bf16-rounded inputs.

Bar: max over outputs of |y - O| / sum|x||w| <= 4.5e-3 (one bf16 rounding of
the output, 2^-8 relative, plus fp32 accumulation; derivation beside TOL in
gpu_util).  Integer-valued inputs must match the oracle's exact sums after the
same single rounding, bit for bit.  Every 16-bit kernel family (column-staged,
row-per-pixel, segment-staged, register-staged) is run with bf16 operands."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import Run, TOL, assert_kernel, check_full, check_sampled, oracle_inputs, rel_err, say
from test_gpu_conv import EDGE, SEG_SHAPES, _id
from paper_2608_20725_amd import workloads

pytestmark = pytest.mark.gpu

BF = torch.bfloat16


def _round_bf16(a):
    """Nearest-even bf16 rounding of exact fp64 values that fp32 holds exactly."""
    return torch.from_numpy(a).to(BF).double().numpy()


@pytest.mark.parametrize("shape", EDGE, ids=_id)
def test_bf16_edge_shapes(shape):
    N, Ci, H, W, Co, Kh, Kw, s = shape
    say("conv bf16", shape)
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=7 + sum(shape))
    run = Run(x, w, s, BF)
    check_full(run, x, w)
    run.check_out_guards()
    run.check_workspace_guard()


@pytest.mark.parametrize("shape", EDGE[-19:], ids=_id)
def test_bf16_integer_inputs_exact(shape):
    """Inputs in {-2..2}: every partial sum is an integer below 2^24, exact in
    fp32 whatever the order; the output is that integer rounded to bf16 once."""
    N, Ci, H, W, Co, Kh, Kw, s = shape
    say("conv bf16 int", shape)
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=11, dist="int2")
    run = Run(x, w, s, BF)
    ref = _round_bf16(oracle.conv(x.double().numpy(), w.double().numpy(), s))
    assert np.array_equal(run.out_np(), ref)


@pytest.mark.parametrize("layer", workloads.ALL, ids=lambda l: l.name)
def test_bf16_layers_small_batch(layer):
    say("conv bf16 N=2", layer.name)
    x, w = workloads.draw_layer(layer, N=min(2, layer.N))
    run = Run(x, w, layer.stride, BF)
    check_full(run, x, w)
    run.check_out_guards()


@pytest.mark.parametrize("layer", workloads.ALL, ids=lambda l: l.name)
def test_bf16_layers_full_batch_sampled(layer):
    """Every configured layer at its full batch: all outputs of images 0 and
    N-1 (when affordable) and 4096 random outputs against the oracle."""
    say("conv bf16 full", layer.name)
    x, w = workloads.draw_layer(layer)
    run = Run(x, w, layer.stride, BF)
    r, n = check_sampled(run, x, w, seed=layer.seed)
    say("  max rel err %.3g over %d outputs" % (r, n))
    run.check_out_guards()


# Each 16-bit kernel family with bf16 operands, forced through the tuning
# variables on shapes that reach it; the row-per-pixel tiles accumulate in the
# same order and must agree bit for bit.
@pytest.mark.parametrize("shape", EDGE[-3:] + [(2, 64, 24, 24, 64, 3, 3, 1)], ids=_id)
def test_bf16_row_kernel_on_column_shapes(shape, monkeypatch):
    N, Ci, H, W, Co, Kh, Kw, s = shape
    say("conv bf16 row kernel", shape)
    monkeypatch.setenv("IM2WIN_FP16_KERNEL", "pipe")
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=13)
    run = Run(x, w, s, BF)
    check_full(run, x, w)
    run.check_out_guards()


@pytest.mark.parametrize("shape", SEG_SHAPES, ids=_id)
def test_bf16_register_kernel_on_segment_shapes(shape, monkeypatch):
    N, Ci, H, W, Co, Kh, Kw, s = shape
    say("conv bf16 register-staged kernel", shape)
    monkeypatch.setenv("IM2WIN_FP16_KERNEL", "regs")
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=19)
    run = Run(x, w, s, BF)
    check_full(run, x, w)
    run.check_out_guards()


BF16_VARIANTS = [
    ("IM2WIN_FP16_TILE", ["c32p128s3", "c64p128s3", "c128p128s2", "c256p256s2w8", "c128p256s2w8"],
     (2, 16, 13, 13, 72, 5, 5, 1), True),
    ("IM2WIN_FP16_COL", ["k3c64p256t32s2", "k3c64p128t32s2", "k3c128p256t16s3", "k3c256p256t32s2w8",
                         "k3c256p192t32s2w8"],
     (2, 64, 24, 24, 300, 3, 3, 1), False),
    ("IM2WIN_FP16_SEG", ["s64p256", "s96p128", "s128p128"], (2, 6, 13, 90, 200, 3, 5, 1), True),
]


@pytest.mark.parametrize("case", BF16_VARIANTS, ids=lambda c: c[0] + "-" + _id(c[2]))
def test_bf16_kernel_variants(case, monkeypatch):
    var, names, shape, same_order = case
    N, Ci, H, W, Co, Kh, Kw, s = shape
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=17)
    first = None
    for name in names:
        say("bf16 variant", var, name, shape)
        monkeypatch.setenv(var, name)
        if var == "IM2WIN_FP16_TILE":
            monkeypatch.setenv("IM2WIN_FP16_KERNEL", "pipe")
        assert_kernel(shape, BF, var, name)
        run = Run(x, w, s, BF)
        check_full(run, x, w)
        out = run.out_np()
        if first is None:
            first = out
        elif same_order:
            assert np.array_equal(out.view(np.uint8), first.view(np.uint8)), name


@pytest.mark.parametrize("Ci", [8, 2], ids=["aligned", "unaligned"])
def test_bf16_round_to_nearest_even(Ci):
    """1x1 conv whose output at pixel p is exactly 1 + t_p 2^-8 (channel 0
    holds 1, channel 1 holds t_p 2^-8, both filter taps 1; every value is a
    bf16 and every sum exact in fp32).  bf16 spacing at 1 is 2^-7, so
    t = 1, 3, 5, 7 are ties, which go to the even neighbour, and t = 1.5 is
    below the midpoint; a truncating or ties-away conversion fails."""
    t = [1.0, 3.0, 5.0, 1.5, 7.0, 1.0, 3.0, 5.0]
    want = {1.0: 1.0, 3.0: 1 + 2.0 ** -6, 5.0: 1 + 2.0 ** -6, 1.5: 1 + 2.0 ** -7, 7.0: 1 + 2.0 ** -5}
    x = torch.zeros(1, 1, len(t), Ci)
    x[0, 0, :, 0] = 1.0
    x[0, 0, :, 1] = torch.tensor(t) * 2.0 ** -8
    w = torch.zeros(1, 1, Ci, 16)
    w[0, 0, 0, :] = 1.0
    w[0, 0, 1, :] = 1.0
    assert torch.equal(x.to(BF).float(), x) and torch.equal(w.to(BF).float(), w)
    run = Run(x, w, 1, BF)
    y = run.out_np()[0, 0]
    for p, tp in enumerate(t):
        assert np.all(y[p] == want[tp]), (p, tp, y[p])


def test_bf16_deterministic():
    layer = workloads.CFG2
    x, w = workloads.draw_layer(layer, N=4)
    run = Run(x, w, layer.stride, BF)
    first = run.out.clone()
    run.rerun_conv()
    assert torch.equal(first.view(torch.int16), run.out.view(torch.int16))


@pytest.mark.parametrize("shape", [(2, 16, 12, 14, 40, 5, 5, 1), (2, 16, 12, 40, 40, 3, 3, 1),
                                   (2, 3, 30, 70, 20, 3, 3, 1)], ids=_id)
def test_bf16_nonfinite_inputs_stay_in_their_windows(shape):
    N, Ci, H, W, Co, Kh, Kw, s = shape
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=23)
    rng = np.random.default_rng(23)
    for v in (float("inf"), float("-inf"), float("nan")):
        x[rng.integers(N), rng.integers(H), rng.integers(W), rng.integers(Ci)] = v
    run = Run(x, w, s, BF)
    xo, wo = oracle_inputs(x, w, BF)
    with np.errstate(invalid="ignore", over="ignore"):
        ref, absref = oracle.conv(xo, wo, s, with_abs=True)
    y = run.out_np()
    fin = np.isfinite(ref)
    assert (~fin).any() and fin.any()
    assert np.array_equal(np.isfinite(y), fin)
    assert rel_err(y[fin], ref[fin], absref[fin]) <= TOL[BF]

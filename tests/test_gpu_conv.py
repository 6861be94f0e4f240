"""fp32 (vector ALU) and fp16 (MFMA, fp32 accumulation) windowed convolution
on the GPU against the fp64 oracle.

Bar: max over outputs of |y - O| / sum|x||w| <= 1e-5 (fp32) and <= 2e-3
(fp16, oracle on the fp16-rounded inputs); where sum|x||w| = 0 the output
must be exactly 0.  Integer-valued inputs must match bit for bit.  Outputs
are NaN-poisoned before each call (every element must be written) and
guarded on both sides (nothing written outside)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_20725_amd as pkg
from gpu_util import Run, TOL, assert_kernel, check_full, check_sampled, oracle_inputs, rel_err, say
from oracle_checks import TINY
from paper_2608_20725_amd import workloads

pytestmark = pytest.mark.gpu

DTYPES = [torch.float32, torch.float16]
DT_IDS = ["f32", "f16"]

# (N, C_i, H, W, C_o, K_h, K_w, s): tiles with ragged tails in pixels, taps
# and channels; C_o below, at and above one wave's 16 channels and the MFMA
# tile sizes; windows that are and are not 16-byte aligned; K_h != K_w;
# s > K; 1x1; filter as large as the input.
EDGE = list(TINY) + [
    (1, 3, 32, 32, 16, 3, 3, 1),      # cfg1 shape
    (2, 8, 17, 19, 10, 3, 2, 1),      # C_o < 16
    (1, 16, 15, 23, 17, 2, 3, 2),     # C_o = 16 + 1
    (3, 4, 13, 11, 33, 3, 3, 1),      # C_o = 32 + 1
    (1, 32, 12, 12, 100, 3, 3, 1),    # C_o = 100
    (2, 24, 9, 9, 130, 3, 3, 2),      # C_o = 128 + 2
    (1, 64, 10, 10, 64, 1, 1, 1),     # 1x1
    (2, 7, 9, 9, 40, 9, 9, 1),        # filter = input: one output pixel per image
    (2, 5, 20, 20, 24, 2, 2, 3),      # s > K
    (1, 12, 30, 30, 48, 5, 4, 2),
    (1, 96, 14, 14, 256, 5, 5, 1),    # cv5-like, K = 2400 (ragged for 64-tap stages)
    (5, 3, 40, 37, 96, 11, 11, 4),    # stem-like, K = 363
    (1, 130, 6, 6, 20, 3, 3, 1),      # K = 1170
    (300, 1, 3, 3, 5, 2, 2, 1),       # many tiny images: tiles span many strips
    # segment-staged fp16 kernel (windows not 16-byte aligned): tiles over
    # several strips and images, taps past K in the last 64-tap stage
    (2, 3, 30, 70, 20, 3, 3, 1),      # tile spans an image boundary
    (1, 5, 19, 150, 100, 5, 5, 2),    # K = 125: second stage ragged; C_o ragged in 128
    (3, 3, 40, 61, 70, 11, 11, 4),    # 11 strips per 128-pixel tile, segments near the LDS limit
    (2, 3, 9, 80, 40, 1, 1, 2),       # s > K_w: window step longer than the window
    (2, 1, 50, 50, 8, 3, 3, 1),       # C_i = 1
    (1, 20, 20, 100, 64, 3, 3, 1),    # C_i = 20: 8-byte aligned windows, K = 180
    (2, 6, 13, 90, 200, 3, 5, 1),     # two channel tiles, the second ragged
    # column-staged fp16 kernel: strip runs inside a tile, taps past K_h*C_i
    # inside the last stage, ragged pixel and channel tiles
    (3, 24, 11, 30, 72, 3, 3, 1),     # K_h*C_i = 72: last stage 8 of 32 taps
    (2, 16, 21, 40, 40, 3, 3, 1),     # K_h*C_i = 48
    (1, 8, 13, 120, 20, 7, 7, 2),     # K_w = 7, stride 2: 2 new columns per pixel
]


def _id(t):
    return "x".join(map(str, t))


@pytest.mark.parametrize("dtype", DTYPES, ids=DT_IDS)
@pytest.mark.parametrize("shape", EDGE, ids=_id)
def test_conv_edge_shapes(shape, dtype):
    N, Ci, H, W, Co, Kh, Kw, s = shape
    say("conv", shape, dtype)
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=7 + sum(shape))
    run = Run(x, w, s, dtype)
    check_full(run, x, w)
    run.check_out_guards()
    run.check_workspace_guard()


@pytest.mark.parametrize("dtype", DTYPES, ids=DT_IDS)
@pytest.mark.parametrize("shape", EDGE[-19:], ids=_id)
def test_conv_integer_inputs_exact(shape, dtype):
    """Inputs in {-2..2}: every partial sum is an integer below 2^24, so any
    summation order gives the exact result."""
    N, Ci, H, W, Co, Kh, Kw, s = shape
    say("conv int", shape, dtype)
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=11, dist="int2")
    run = Run(x, w, s, dtype)
    ref = oracle.conv(x.double().numpy(), w.double().numpy(), s)
    if dtype == torch.float16:
        ref = ref.astype(np.float16).astype(np.float64)   # the one rounding on store
    assert np.array_equal(run.out_np(), ref)


@pytest.mark.parametrize("dtype", DTYPES, ids=DT_IDS)
@pytest.mark.parametrize("layer", workloads.ALL, ids=lambda l: l.name)
def test_conv_layers_small_batch(layer, dtype):
    """Every configured layer shape with batch 2, all outputs checked."""
    say("conv N=2", layer.name, dtype)
    x, w = workloads.draw_layer(layer, N=min(2, layer.N))
    run = Run(x, w, layer.stride, dtype)
    check_full(run, x, w)
    run.check_out_guards()


@pytest.mark.parametrize("dtype", DTYPES, ids=DT_IDS)
@pytest.mark.parametrize("layer", workloads.ALL, ids=lambda l: l.name)
def test_conv_layers_full_batch_sampled(layer, dtype):
    """Every configured layer at its full batch, in the launch configuration
    the benchmark times: all outputs of images 0 and N-1 (when affordable) and
    4096 random outputs, each against the oracle."""
    say("conv full", layer.name, dtype, pkg.conv_im2win_kernel_name(
        layer.N, layer.C_i, layer.H, layer.W, layer.C_o, layer.K_h, layer.K_w, layer.stride, dtype))
    x, w = workloads.draw_layer(layer)
    run = Run(x, w, layer.stride, dtype)
    r, n = check_sampled(run, x, w, seed=layer.seed)
    say("  max rel err %.3g over %d outputs" % (r, n))
    run.check_out_guards()
    # run-to-run determinism at full size: the same bits again
    first = run.out.clone()
    run.rerun_conv()
    bits = torch.int16 if dtype == torch.float16 else torch.int32
    assert torch.equal(first.view(bits), run.out.view(bits))


@pytest.mark.parametrize("dtype", DTYPES, ids=DT_IDS)
def test_conv_deterministic(dtype):
    layer = workloads.CFG2
    say("determinism", dtype)
    x, w = workloads.draw_layer(layer, N=4)
    run = Run(x, w, layer.stride, dtype)
    first = run.out.clone()
    run.rerun_conv()
    assert torch.equal(first.view(torch.int16 if dtype == torch.float16 else torch.int32),
                       run.out.view(torch.int16 if dtype == torch.float16 else torch.int32))


@pytest.mark.parametrize("dtype", DTYPES, ids=DT_IDS)
def test_conv_on_side_stream(dtype):
    shape = (3, 16, 14, 14, 48, 3, 3, 1)
    N, Ci, H, W, Co, Kh, Kw, s = shape
    say("side stream", dtype)
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=5)
    st = torch.cuda.Stream()
    with torch.cuda.stream(st):
        run = Run(x, w, s, dtype, stream=st)
    st.synchronize()
    check_full(run, x, w)


def test_fp16_rounding_once():
    """Output rounding: the fp16 result of a dot product whose exact value is
    representable is that value."""
    x = torch.zeros(1, 1, 1, 64)
    w = torch.zeros(1, 1, 64, 16)
    x[0, 0, 0, :] = torch.arange(64) % 5 - 2
    w[0, 0, :, :] = (torch.arange(64 * 16).reshape(64, 16) % 7 - 3).float()
    run = Run(x, w, 1, torch.float16)
    ref = oracle.conv(x.double().numpy(), w.double().numpy(), 1)
    assert np.array_equal(run.out_np(), ref)


# The fp16 path has two kernels: windows staged per input column (the
# default for K_w in {3, 7} with C_o <= 128, when a tile's columns fit) and
# windows staged per pixel row (every other layer).  IM2WIN_FP16_KERNEL=pipe
# forces the second, so both are checked on the shapes that select the first.
@pytest.mark.parametrize("shape", EDGE[-3:] + [(2, 64, 24, 24, 64, 3, 3, 1)], ids=_id)
def test_fp16_row_kernel_on_column_shapes(shape, monkeypatch):
    N, Ci, H, W, Co, Kh, Kw, s = shape
    say("conv fp16 row kernel", shape)
    monkeypatch.setenv("IM2WIN_FP16_KERNEL", "pipe")
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=13)
    run = Run(x, w, s, torch.float16)
    check_full(run, x, w)
    run.check_out_guards()


# Windows that are not 16-byte aligned (C_i not a multiple of 8) go to the
# segment-staged fp16 kernel when a tile's strip segments fit in LDS, else to
# the register-staged one; IM2WIN_FP16_KERNEL=regs forces the latter, so both
# are checked on the shapes that select the former.
SEG_SHAPES = [(1, 3, 32, 32, 16, 3, 3, 1), (2, 3, 30, 70, 20, 3, 3, 1), (3, 3, 40, 61, 70, 11, 11, 4),
              (2, 6, 13, 90, 200, 3, 5, 1)]


@pytest.mark.parametrize("shape", SEG_SHAPES, ids=_id)
def test_fp16_register_kernel_on_segment_shapes(shape, monkeypatch):
    N, Ci, H, W, Co, Kh, Kw, s = shape
    say("conv fp16 register-staged kernel", shape)
    monkeypatch.setenv("IM2WIN_FP16_KERNEL", "regs")
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=19)
    run = Run(x, w, s, torch.float16)
    check_full(run, x, w)
    run.check_out_guards()


# Every kernel variant the launchers can pick (by layer or through the tuning
# variables), on shapes that reach it: each must match the oracle, and where
# the variants of a kernel accumulate K in the same order (the row-per-pixel
# fp16 tiles, the fp32 kernels) each other bit for bit.  The names mirror the
# variant tables in the C++ sources.
VARIANT_CASES = [
    # (environment variable, names, shape, dtype, same summation order)
    ("IM2WIN_FP16_TILE", ["c32p128s3", "c64p128s3", "c128p128s2", "c256p256s2w8", "c128p256s2w8", "c128p128s1"],
     (2, 16, 13, 13, 72, 5, 5, 1), torch.float16, True),
    # the register-staged kernel forced on 16-byte-aligned windows (its filter
    # pack follows): the same summation order as the row-per-pixel kernel
    ("IM2WIN_FP16_KERNEL", ["pipe", "regs"], (2, 16, 13, 13, 72, 5, 5, 1), torch.float16, True),
    ("IM2WIN_FP16_KERNEL", ["pipe", "regs"], (1, 64, 20, 20, 300, 3, 3, 1), torch.float16, True),
    ("IM2WIN_FP16_COL", ["k3c64p256t32s2", "k3c64p128t32s2", "k3c128p256t16s3", "k3c256p256t32s2w8",
                         "k3c256p192t32s2w8", "k3c128p128t32s2"],
     (2, 64, 24, 24, 300, 3, 3, 1), torch.float16, False),
    # the 7x7 column-staged tiles (filter width 7, stride 1 and 2)
    ("IM2WIN_FP16_COL", ["k7c64p256t16s3", "k7c64p128t16s2", "k7c64p256t32s2"],
     (2, 16, 19, 40, 70, 7, 7, 1), torch.float16, False),
    ("IM2WIN_FP16_COL", ["k7c64p256t16s3", "k7c64p128t16s2", "k7c64p256t32s2"],
     (2, 8, 23, 121, 40, 7, 7, 2), torch.float16, False),
    ("IM2WIN_FP32_KERNEL", ["p8c8l8s2k16", "p6c8l8s2k16", "p4c8l8s2k16", "p4c16l1s2k16", "p8c8l8s2k16g4",
                            "p4c12l8s2k16", "p8c12l8s2k16", "p4c12l8s2k16g4", "p8c12l8s2k16g4", "regs"],
     (2, 16, 17, 19, 100, 3, 3, 1), torch.float32, True),
    ("IM2WIN_FP32_KERNEL", ["p8c8l8s2k16g4", "p6c8l8s2k16g4", "p4c8l8s2k16g4", "p4c12l8s2k16g4", "p8c12l8s2k16g4",
                            "regs"],
     (3, 3, 40, 61, 70, 11, 11, 4), torch.float32, True),
    # 96-channel tiles: C_o = 96 exactly and C_o = 200 (a ragged third tile)
    ("IM2WIN_FP32_KERNEL", ["p8c8l8s2k16", "p4c12l8s2k16", "p8c12l8s2k16", "regs"],
     (2, 8, 20, 22, 96, 3, 3, 1), torch.float32, True),
    ("IM2WIN_FP32_KERNEL", ["p8c8l8s2k16g4", "p4c12l8s2k16g4", "regs"], (2, 3, 30, 29, 200, 5, 5, 2), torch.float32,
     True),
    # taps split over the waves: another summation order, K = 144 ragged in
    # 64-tap stages
    ("IM2WIN_FP32_KERNEL", ["p8c8l8s2k16t4", "p4c8l8s2k16t4", "p4c8l8s2k16t4w8"], (2, 16, 17, 19, 100, 3, 3, 1),
     torch.float32, True),
    ("IM2WIN_FP16_SEG", ["s64p256", "s96p128", "s128p128"], (2, 6, 13, 90, 200, 3, 5, 1), torch.float16,
     True),
]


@pytest.mark.parametrize("case", VARIANT_CASES, ids=lambda c: c[0] + "-" + _id(c[2]))
def test_kernel_variants_agree(case, monkeypatch):
    var, names, shape, dtype, same_order = case
    N, Ci, H, W, Co, Kh, Kw, s = shape
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=17)
    first = None
    for name in names:
        say("variant", var, name, shape)
        monkeypatch.setenv(var, name)
        if var == "IM2WIN_FP16_TILE":
            monkeypatch.setenv("IM2WIN_FP16_KERNEL", "pipe")
        assert_kernel(shape, dtype, var, name)
        run = Run(x, w, s, dtype)
        check_full(run, x, w)
        out = run.out_np()
        if first is None:
            first = out
        elif same_order:
            assert np.array_equal(out.view(np.uint8), first.view(np.uint8)), name



# Differential check of the load rings: each ring kernel against the same
# tile with its ring serialized (a stage's loads issued only after every wave
# has finished with the previous one, and waited for in full, so nothing is
# in flight while LDS is read).  Both compute the same sums in the same
# order, so a missing wait or barrier in the ring would show as a bit
# difference.  Shapes with many stages and many tiles per CU.
SERIAL_CASES = [
    # (variable, ring variant, shape, dtype)
    ("IM2WIN_FP16_COL", "k3c64p128t32s2", (8, 64, 56, 56, 64, 3, 3, 1), torch.float16),
    ("IM2WIN_FP16_COL", "k7c64p256t16s3", (2, 64, 60, 120, 64, 7, 7, 2), torch.float16),
    ("IM2WIN_FP16_COL", "k3c256p192t32s2w8", (16, 512, 14, 14, 512, 3, 3, 1), torch.bfloat16),
    ("IM2WIN_FP16_SEG", "s64p256", (8, 3, 100, 100, 64, 3, 3, 1), torch.float16),
    ("IM2WIN_FP32_KERNEL", "p8c8l8s2k16", (8, 64, 56, 56, 64, 3, 3, 1), torch.float32),
    ("IM2WIN_FP32_KERNEL", "p6c8l8s2k16g4", (8, 3, 100, 100, 64, 7, 7, 2), torch.float32),
    ("IM2WIN_FP32_KERNEL", "p4c8l8s2k16t4", (16, 256, 14, 14, 256, 3, 3, 1), torch.float32),
    ("IM2WIN_FP32_KERNEL", "p4c8l8s2k16t4w8", (16, 256, 14, 14, 256, 3, 3, 1), torch.float32),
]


@pytest.mark.parametrize("case", SERIAL_CASES, ids=lambda c: c[1] + "-" + _id(c[2]))
def test_ring_matches_serialized_ring(case, monkeypatch):
    var, name, shape, dtype = case
    N, Ci, H, W, Co, Kh, Kw, s = shape
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=53)
    outs = []
    for v in (name, name + "-serial"):
        monkeypatch.setenv(var, v)
        say("ring", v, shape, dtype)
        assert_kernel(shape, dtype, var, v)
        run = Run(x, w, s, dtype)
        if not outs:
            check_sampled(run, x, w, seed=3)
        run.check_out_guards()
        outs.append(run.out.clone())
    bits = torch.int32 if dtype == torch.float32 else torch.int16
    assert torch.equal(outs[0].view(bits), outs[1].view(bits))


# Persistent launch of the column-staged kernel (one round of workgroups
# walking the tiles) against one workgroup per tile: the same sums in the
# same order per tile, so bit-identical outputs.  Shapes with more tiles than
# one round holds, so that the persistent loop runs; the oracle checks one.
PERSIST_CASES = [
    ("k3c64p128t32s2", (64, 64, 56, 56, 64, 3, 3, 1), torch.float16),
    ("k3c64p256t32s2", (16, 64, 112, 112, 128, 3, 3, 1), torch.float16),
    ("k3c128p128t32s2", (16, 64, 112, 112, 128, 3, 3, 1), torch.bfloat16),
    ("k7c64p256t32s2", (8, 64, 224, 224, 64, 7, 7, 2), torch.bfloat16),
    ("k3c256p192t32s2w8", (256, 512, 14, 14, 512, 3, 3, 1), torch.float16),
]


@pytest.mark.parametrize("case", PERSIST_CASES, ids=lambda c: c[0])
def test_persistent_column_launch_same_bits(case, monkeypatch):
    name, shape, dtype = case
    N, Ci, H, W, Co, Kh, Kw, s = shape
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=61)
    monkeypatch.setenv("IM2WIN_FP16_COL", name)
    outs = []
    for mode in ("on", "off"):
        monkeypatch.setenv("IM2WIN_FP16_PERSIST", mode)
        say("persist", mode, name, shape, dtype)
        assert_kernel(shape, dtype, "IM2WIN_FP16_COL", name)
        run = Run(x, w, s, dtype)
        if not outs:
            check_sampled(run, x, w, seed=5)
        run.check_out_guards()
        outs.append(run.out.clone())
    assert torch.equal(outs[0].view(torch.int16), outs[1].view(torch.int16))


# The K-loop tap order (IM2WIN_TAP_ORDER): linear, or column slices of one
# tap range in turn (columns grouped by residue mod the stride).  Both are fixed orders that the oracle bounds; the
# DMA-staged fp32 kernel (column by default) and the register-staged one
# follow the same order, so they agree bit for bit in either.
TAP_CASES = [
    # (shape, dtype, forced variables)
    ((2, 16, 17, 19, 100, 3, 3, 1), torch.float32, {"IM2WIN_FP32_KERNEL": "p8c8l8s2k16"}),
    ((2, 16, 23, 41, 40, 7, 7, 2), torch.float32, {"IM2WIN_FP32_KERNEL": "p4c12l8s2k16"}),
    # stride 2, K_h*C_i a multiple of 32: columns 0, 2, 4, 6, 1, 3, 5 in turn
    ((2, 32, 23, 41, 40, 7, 7, 2), torch.float32, {"IM2WIN_FP32_KERNEL": "p8c8l8s2k16"}),
    ((2, 64, 23, 41, 72, 5, 5, 2), torch.float16, {"IM2WIN_FP16_KERNEL": "pipe"}),
    ((2, 64, 14, 14, 200, 3, 3, 1), torch.float32, {"IM2WIN_FP32_KERNEL": "p4c8l8s2k16t4"}),
    ((2, 64, 20, 20, 96, 3, 3, 1), torch.float16, {"IM2WIN_FP16_KERNEL": "pipe"}),
    ((2, 64, 20, 20, 200, 5, 5, 2), torch.bfloat16, {"IM2WIN_FP16_TILE": "c128p128s1"}),
]


@pytest.mark.parametrize("case", TAP_CASES, ids=lambda c: _id(c[0]) + "-" + str(c[1])[6:])
def test_tap_orders(case, monkeypatch):
    shape, dtype, env = case
    N, Ci, H, W, Co, Kh, Kw, s = shape
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=59)
    for k, v in env.items():
        monkeypatch.setenv(k, v)
    bits = torch.int32 if dtype == torch.float32 else torch.int16
    for order in ("linear", "column"):
        monkeypatch.setenv("IM2WIN_TAP_ORDER", order)
        say("tap order", order, shape, dtype, env)
        run = Run(x, w, s, dtype)
        check_full(run, x, w)
        run.check_out_guards()
        if env.get("IM2WIN_FP32_KERNEL", "").endswith("k16"):
            # the register-staged kernel sums in the same order as the
            # DMA-staged ones that do not split a stage's taps
            first = run.out.clone()
            monkeypatch.setenv("IM2WIN_FP32_KERNEL", "regs")
            run2 = Run(x, w, s, dtype)
            monkeypatch.setenv("IM2WIN_FP32_KERNEL", env["IM2WIN_FP32_KERNEL"])
            assert torch.equal(first.view(bits), run2.out.view(bits))


# The XCD-aware tile order (several channel tiles) against launch order
# (IM2WIN_TILE_ORDER=linear): each tile computes the same sums whichever
# workgroup takes it, so the outputs agree bit for bit.  Grids with a ragged
# share per XCD (tiles not a multiple of 8) and with fewer tiles than XCDs.
ORDER_CASES = [
    # (forced variables, shape, dtype, matrix-core fp32)
    ({}, (2, 16, 17, 19, 300, 3, 3, 1), torch.float32, False),
    ({"IM2WIN_FP32_KERNEL": "p4c8l8s2k16t4"}, (2, 16, 17, 19, 300, 3, 3, 1), torch.float32, False),
    ({"IM2WIN_FP32_KERNEL": "p4c8l8s2k16t4w8"}, (2, 16, 17, 19, 300, 3, 3, 1), torch.float32, False),
    ({}, (1, 8, 6, 6, 200, 3, 3, 1), torch.float32, False),
    ({}, (2, 64, 24, 24, 300, 3, 3, 1), torch.float32, True),
    ({}, (1, 8, 6, 6, 200, 3, 3, 1), torch.float32, True),
    ({}, (2, 64, 24, 24, 300, 3, 3, 1), torch.float16, False),
    ({"IM2WIN_FP16_KERNEL": "pipe"}, (2, 16, 13, 13, 300, 5, 5, 1), torch.float16, False),
    ({"IM2WIN_FP16_KERNEL": "regs"}, (2, 16, 13, 13, 300, 5, 5, 1), torch.bfloat16, False),
    ({}, (1, 8, 6, 6, 200, 3, 3, 1), torch.float16, False),
]


@pytest.mark.parametrize("case", ORDER_CASES,
                         ids=lambda c: "-".join(list(c[0].values()) + [_id(c[1]), str(c[2])[6:]] + (["mfma"] if c[3] else [])))
def test_tile_order_same_bits(case, monkeypatch):
    env, shape, dtype, mfma = case
    N, Ci, H, W, Co, Kh, Kw, s = shape
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=19)
    for k, v in env.items():
        monkeypatch.setenv(k, v)
    outs = []
    for order in ("xcd", "linear"):
        say("tile order", order, env, shape, dtype)
        if order == "linear":
            monkeypatch.setenv("IM2WIN_TILE_ORDER", "linear")
        run = Run(x, w, s, dtype, conv=not mfma)
        if mfma:
            pkg.conv_im2win_fp32_mfma(run.ws, run.wd, run.out, run.N, run.Ci, run.H, run.W, s)
            torch.cuda.synchronize()
        check_full(run, x, w)
        run.check_out_guards()
        outs.append(run.out.clone())
    bits = torch.int32 if dtype == torch.float32 else torch.int16
    assert torch.equal(outs[0].view(bits), outs[1].view(bits))


# Non-finite inputs stay inside the windows that hold them: an output is
# finite exactly where the oracle's is (a kernel that multiplied the zero
# filter padding past K by a neighbouring window's Inf would turn an
# unrelated output into NaN), and the finite outputs meet the usual bar.
# One shape per kernel path: fp32 DMA-staged and register-staged, fp16
# pixel-row, column, segment and register-staged.
NONFINITE_CASES = [
    ((2, 16, 12, 14, 40, 3, 3, 1), torch.float32),
    ((2, 3, 12, 14, 40, 3, 3, 1), torch.float32),
    ((2, 16, 12, 14, 40, 5, 5, 1), torch.float16),
    ((2, 16, 12, 40, 40, 3, 3, 1), torch.float16),
    ((2, 3, 30, 70, 20, 3, 3, 1), torch.float16),
    ((1, 12, 30, 30, 48, 5, 4, 2), torch.float16),
]


@pytest.mark.parametrize("case", NONFINITE_CASES, ids=lambda c: _id(c[0]) + ("-f32" if c[1] == torch.float32 else "-f16"))
def test_nonfinite_inputs_stay_in_their_windows(case):
    shape, dtype = case
    N, Ci, H, W, Co, Kh, Kw, s = shape
    say("non-finite", shape, dtype)
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=23)
    rng = np.random.default_rng(23)
    for v in (float("inf"), float("-inf"), float("inf"), float("nan")):
        x[rng.integers(N), rng.integers(H), rng.integers(W), rng.integers(Ci)] = v
    run = Run(x, w, s, dtype)
    xo, wo = oracle_inputs(x, w, dtype)
    with np.errstate(invalid="ignore", over="ignore"):
        ref, absref = oracle.conv(xo, wo, s, with_abs=True)
    y = run.out_np()
    fin = np.isfinite(ref)
    assert (~fin).any() and fin.any()
    assert np.array_equal(np.isfinite(y), fin), "%d outputs differ in finiteness" % int(
        (np.isfinite(y) != fin).sum())
    r = rel_err(y[fin], ref[fin], absref[fin])
    assert r <= TOL[dtype], "max |err|/sum|x||w| = %.3g" % r
    run.check_out_guards()


# The column-staged fp32 kernel (IM2WIN_FP32_COLS; each distinct input column
# of a tile loaded once per tap block): every output against the oracle on
# shapes with several strip runs per tile, ragged pixel and channel tiles, a
# tap block cut by T = K_h*C_i, and stride 2; its serialized ring gives the
# same bits.
COLS32_CASES = [
    ("k3p256t16", (2, 8, 19, 23, 72, 3, 3, 1)),     # T = 24: the second 16-tap block half used
    ("k3p128t16", (3, 4, 9, 40, 130, 3, 3, 1)),     # three channel tiles, the last of 2
    ("k3p256t8", (2, 12, 30, 17, 64, 3, 3, 1)),     # 15 output columns per strip: many runs per tile
    ("k5p256t8", (2, 16, 14, 20, 40, 5, 5, 1)),
    ("k7p256t8", (2, 8, 23, 121, 40, 7, 7, 2)),
    ("k7p128t8", (1, 4, 20, 60, 64, 7, 7, 1)),
]


@pytest.mark.parametrize("case", COLS32_CASES, ids=lambda c: c[0] + "-" + _id(c[1]))
def test_fp32_column_kernel(case, monkeypatch):
    name, shape = case
    N, Ci, H, W, Co, Kh, Kw, s = shape
    say("fp32 column-staged", name, shape)
    monkeypatch.setenv("IM2WIN_FP32_COLS", name)
    assert_kernel(shape, "f32", "IM2WIN_FP32_COLS", name)
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=41)
    run = Run(x, w, s, torch.float32)
    check_full(run, x, w)
    run.check_out_guards()
    run.check_workspace_guard()
    if name == "k3p256t16":
        monkeypatch.setenv("IM2WIN_FP32_COLS", name + "-serial")
        twin = Run(x, w, s, torch.float32)
        assert torch.equal(run.out.view(torch.int32), twin.out.view(torch.int32))

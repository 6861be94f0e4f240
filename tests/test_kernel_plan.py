"""Kernel choice on the host: conv_im2win_kernel_name reports the kernel a
conv call runs, the tuning variables are checked (an unknown name, a
contradiction, or a forced kernel that cannot run the layer is refused with
IM2WIN_EINVAL by the query and by every call), and the mini-batch path's
plan holds for a smaller last chunk.  No call here reaches a GPU."""
import os

import pytest

import paper_2608_20725_amd as pkg
from paper_2608_20725_amd import workloads

EINVAL = -1
VARS = ("IM2WIN_FP16_KERNEL", "IM2WIN_FP16_COL", "IM2WIN_FP16_TILE", "IM2WIN_FP16_SEG", "IM2WIN_FP32_KERNEL",
        "IM2WIN_FP32_TILE", "IM2WIN_FP32_MFMA_TILE", "IM2WIN_TRANSFORM_ORDER", "IM2WIN_TILE_ORDER",
        "IM2WIN_TAP_ORDER", "IM2WIN_FP16_SPLIT", "IM2WIN_FP32_COLS", "IM2WIN_TRANSFORM_KERNEL",
        "IM2WIN_FP16_PERSIST")


@pytest.fixture(autouse=True)
def clean_env(monkeypatch):
    for v in VARS:
        monkeypatch.delenv(v, raising=False)
    if not os.path.exists(pkg.library_path()):
        from paper_2608_20725_amd import build
        build.build()


def name(shape, dt, **kw):
    N, Ci, H, W, Co, Kh, Kw, s = shape
    return pkg.conv_im2win_kernel_name(N, Ci, H, W, Co, Kh, Kw, s, dt, **kw)


def status(shape, dt, **kw):
    try:
        name(shape, dt, **kw)
        return 0
    except pkg.Im2winError as e:
        return e.status


def lay(l):
    return (l.N, l.C_i, l.H, l.W, l.C_o, l.K_h, l.K_w, l.stride)


@pytest.mark.parametrize("layer", workloads.ALL, ids=lambda l: l.name)
def test_every_layer_has_a_plan(layer):
    sh = lay(layer)
    aligned16 = layer.C_i % 8 == 0
    f16 = name(sh, "f16")
    assert f16 == name(sh, "bf16")  # same kernels for both 16-bit operand types
    fam = f16.split()[0]
    assert fam in (("conv_fp16_col", "conv_fp16_pipe") if aligned16 else
                   ("conv_fp16_stem", "conv_fp16_seg", "conv_fp16_kernel"))
    f32 = name(sh, "f32")
    assert f32.split()[0] in ("conv_fp32_dma", "conv_fp32_kernel", "conv_fp32_stem")
    if layer.C_i % 4 == 0:
        assert name(sh, "f32", fp32_matrix_cores=True).startswith("conv_fp32_mfma ")
    else:   # the matrix-core fp32 kernel needs 16-byte window chunks
        assert name(sh, "f32", fp32_matrix_cores=True) == f32


@pytest.mark.parametrize("var,value", [(v, "no-such-kernel") for v in VARS] + [("IM2WIN_FP16_KERNEL", "col")])
def test_unknown_tuning_value_refused(monkeypatch, var, value):
    monkeypatch.setenv(var, value)
    for dt in ("f32", "f16"):
        assert status((1, 64, 10, 10, 64, 3, 3, 1), dt) == EINVAL


@pytest.mark.parametrize("env", [
    {"IM2WIN_FP16_COL": "k3c64p128t32s2", "IM2WIN_FP16_KERNEL": "pipe"},
    {"IM2WIN_FP16_COL": "k3c64p128t32s2", "IM2WIN_FP16_SEG": "s64p256"},
    {"IM2WIN_FP16_TILE": "c64p128s3", "IM2WIN_FP16_KERNEL": "regs"},
    {"IM2WIN_FP32_KERNEL": "p8c8l8s2k16", "IM2WIN_FP32_TILE": "m4n16f"},
], ids=lambda e: "+".join(e))
def test_contradictory_tuning_refused(monkeypatch, env):
    for k, v in env.items():
        monkeypatch.setenv(k, v)
    assert status((1, 64, 10, 10, 64, 3, 3, 1), "f16") == EINVAL


@pytest.mark.parametrize("env,shape,dt", [
    # a 7-wide column kernel on a 3x3 layer
    ({"IM2WIN_FP16_COL": "k7c64p128t16s2"}, (1, 64, 10, 10, 64, 3, 3, 1), "f16"),
    # column kernels need 16-byte-aligned windows
    ({"IM2WIN_FP16_COL": "k3c64p128t32s2"}, (1, 3, 10, 10, 64, 3, 3, 1), "f16"),
    # a tile whose distinct columns exceed the kernel's row budget: 7x7
    # stride 2 with 7 output columns per strip, 128-pixel tiles touch 20
    # strips and need 356 of 288 rows
    ({"IM2WIN_FP16_COL": "k7c64p128t16s2"}, (2, 8, 23, 20, 40, 7, 7, 2), "f16"),
    # the row-per-pixel kernels need 16-byte-aligned windows
    ({"IM2WIN_FP16_KERNEL": "pipe"}, (1, 3, 10, 10, 64, 3, 3, 1), "f16"),
    ({"IM2WIN_FP16_TILE": "c64p128s3"}, (1, 3, 10, 10, 64, 3, 3, 1), "f16"),
    # the segment kernel is for unaligned windows only
    ({"IM2WIN_FP16_SEG": "s64p256"}, (1, 64, 10, 10, 64, 3, 3, 1), "f16"),
    # 16-byte DMA windows need C_i % 4 == 0
    ({"IM2WIN_FP32_KERNEL": "p8c8l8s2k16"}, (1, 3, 10, 10, 64, 3, 3, 1), "f32"),
], ids=lambda x: x if isinstance(x, str) else "x".join(map(str, x)) if isinstance(x, tuple) else "+".join(x.values()))
def test_forced_kernel_that_cannot_run_refused(monkeypatch, env, shape, dt):
    for k, v in env.items():
        monkeypatch.setenv(k, v)
    assert status(shape, dt) == EINVAL


def test_forced_mfma_tile_on_unaligned_layer_refused(monkeypatch):
    monkeypatch.setenv("IM2WIN_FP32_MFMA_TILE", "c128p128s2")
    assert status((1, 3, 10, 10, 64, 3, 3, 1), "f32", fp32_matrix_cores=True) == EINVAL
    # the vector-ALU entry point ignores it
    assert name((1, 3, 10, 10, 64, 3, 3, 1), "f32").startswith("conv_fp32_stem ")


@pytest.mark.parametrize("var,value,expect", [
    ("IM2WIN_FP16_KERNEL", "pipe", "conv_fp16_pipe "),
    ("IM2WIN_FP16_KERNEL", "regs", "conv_fp16_kernel "),
    ("IM2WIN_FP16_TILE", "c128p128s1", "conv_fp16_pipe c128p128s1"),
    ("IM2WIN_FP16_COL", "k3c64p256t32s2", "conv_fp16_col k3c64p256t32s2"),
    ("IM2WIN_FP32_KERNEL", "regs", "conv_fp32_kernel m4n16f"),
    ("IM2WIN_FP32_KERNEL", "p4c12l8s2k16", "conv_fp32_dma p4c12l8s2k16"),
    ("IM2WIN_FP32_TILE", "m8n16f", "conv_fp32_kernel m8n16f"),
])
def test_forced_kernel_is_reported(monkeypatch, var, value, expect):
    monkeypatch.setenv(var, value)
    dt = "f32" if "FP32" in var else "f16"
    assert name((2, 64, 24, 24, 64, 3, 3, 1), dt).startswith(expect)


def test_orders_accept_both_names(monkeypatch):
    for v in ("linear", "xcd"):
        monkeypatch.setenv("IM2WIN_TILE_ORDER", v)
        monkeypatch.setenv("IM2WIN_TRANSFORM_ORDER", v)
        assert name((1, 64, 10, 10, 64, 3, 3, 1), "f16")
    for v in ("linear", "column"):
        monkeypatch.setenv("IM2WIN_TAP_ORDER", v)
        assert name((1, 64, 10, 10, 64, 3, 3, 1), "f32")
    monkeypatch.setenv("IM2WIN_TAP_ORDER", "xcd")   # the tile orders' word is not a tap order
    assert status((1, 64, 10, 10, 64, 3, 3, 1), "f32") == EINVAL


def test_transform_kernel_names(monkeypatch):
    """IM2WIN_TRANSFORM_KERNEL takes pieces or gather; any other word is
    refused by every call, the query included."""
    for v in ("pieces", "gather", ""):
        monkeypatch.setenv("IM2WIN_TRANSFORM_KERNEL", v)
        assert name((1, 3, 32, 32, 16, 3, 3, 1), "f16")
    monkeypatch.setenv("IM2WIN_TRANSFORM_KERNEL", "vec")
    assert status((1, 3, 32, 32, 16, 3, 3, 1), "f16") == EINVAL


def test_persist_switch_names(monkeypatch):
    for v in ("on", "off", ""):
        monkeypatch.setenv("IM2WIN_FP16_PERSIST", v)
        assert name((1, 64, 10, 10, 64, 3, 3, 1), "f16")
    monkeypatch.setenv("IM2WIN_FP16_PERSIST", "yes")
    assert status((1, 64, 10, 10, 64, 3, 3, 1), "f16") == EINVAL


# The mini-batch path makes its plan for a full chunk and runs it on the
# smaller last chunk too; the shapes below are ones where a standalone call
# on the last chunk would pick another kernel (and, for the 16-bit path,
# another packed-filter layout), the case the single plan exists for.
@pytest.mark.parametrize("shape,n_chunk,dt", [
    ((160, 512, 14, 14, 512, 3, 3, 1), 128, "f16"),
    ((160, 512, 14, 14, 512, 3, 3, 1), 128, "bf16"),
    ((128, 64, 56, 56, 64, 3, 3, 1), 100, "f32"),
])
def test_chunk_plan_differs_from_last_chunk_standalone(shape, n_chunk, dt):
    N = shape[0]
    last = N - (N // n_chunk) * n_chunk
    full_chunk = name((n_chunk,) + shape[1:], dt)
    last_alone = name((last,) + shape[1:], dt)
    assert full_chunk != last_alone, (full_chunk, last_alone)


@pytest.mark.parametrize("value", ["0", "9", "-1", "2x", "1.5"])
def test_split_out_of_range_refused(monkeypatch, value):
    monkeypatch.setenv("IM2WIN_FP16_SPLIT", value)
    assert status((1, 64, 10, 10, 128, 3, 3, 1), "f16") == EINVAL


def test_split_reported_and_refused_where_it_cannot_run(monkeypatch):
    sh = (2, 64, 24, 24, 128, 3, 3, 1)   # K = 576: 9 stages of 64 taps
    # the layer's default kernel is column-staged: no K split there
    assert name(sh, "f16").startswith("conv_fp16_col ")
    monkeypatch.setenv("IM2WIN_FP16_SPLIT", "3")
    assert status(sh, "f16") == EINVAL
    monkeypatch.setenv("IM2WIN_FP16_TILE", "c128p128s2")
    assert name(sh, "f16") == "conv_fp16_pipe c128p128s2 k3"
    assert name(sh, "bf16") == "conv_fp16_pipe c128p128s2 k3"
    monkeypatch.setenv("IM2WIN_FP16_SPLIT", "1")
    assert name(sh, "f16") == "conv_fp16_pipe c128p128s2"
    # one 64-tap stage cannot be split in two
    monkeypatch.setenv("IM2WIN_FP16_SPLIT", "2")
    assert status((1, 64, 10, 10, 128, 1, 1, 1), "f16") == EINVAL
    # 9 stages in 8 ranges of 2 leave the last range empty
    monkeypatch.setenv("IM2WIN_FP16_SPLIT", "8")
    assert status(sh, "f16") == EINVAL
    # fp32 ignores the 16-bit split
    assert name(sh, "f32").startswith("conv_fp32_dma ")


@pytest.mark.parametrize("layer", workloads.ALL, ids=lambda l: l.name)
def test_default_plan_workspace_not_above_im2col_by_the_split(layer):
    # a K split the planner makes by default keeps the whole 16-bit workspace
    # within the layer's im2col matrix
    sh = lay(layer)
    n = name(sh, "f16")
    if n.split()[-1].startswith("k") and n.split()[0] == "conv_fp16_pipe":
        ws = pkg.conv_workspace_bytes(*sh, "f16")
        assert ws <= pkg.conv_im2col_bytes(sh[0], sh[1], sh[2], sh[3], sh[5], sh[6], sh[7], "f16")


@pytest.mark.parametrize("shape,want", [
    ((2, 3, 224, 224, 64, 3, 3, 1), "conv_fp16_stem m2k2"),     # 27 taps: the default
    ((2, 3, 30, 30, 128, 4, 4, 1), "conv_fp16_stem m4k4"),      # 48 taps, 128 channels
    ((2, 3, 227, 227, 64, 7, 7, 2), "conv_fp16_seg "),          # 147 taps: segment-staged
    ((2, 3, 30, 30, 20, 3, 3, 1), "conv_fp16_seg "),            # C_o not a multiple of 8
    ((2, 3, 30, 30, 136, 3, 3, 1), "conv_fp16_seg "),           # C_o > 128
])
def test_stem_default(shape, want):
    assert name(shape, "f16").startswith(want)


def test_stem_forced(monkeypatch):
    monkeypatch.setenv("IM2WIN_FP16_KERNEL", "stem")
    assert name((2, 3, 227, 227, 64, 7, 7, 2), "f16") == "conv_fp16_stem m2k10"   # up to 160 taps
    assert status((2, 3, 227, 227, 96, 11, 11, 4), "f16") == EINVAL               # 363 taps
    assert status((2, 64, 20, 20, 64, 3, 3, 1), "f16") == EINVAL                  # aligned windows
    assert status((2, 3, 30, 30, 20, 3, 3, 1), "f16") == EINVAL                   # C_o % 8


@pytest.mark.parametrize("shape,want", [
    ((2, 3, 224, 224, 64, 3, 3, 1), "conv_fp32_stem k27"),
    ((2, 3, 30, 30, 16, 2, 2, 1), "conv_fp32_stem k16"),
    ((2, 5, 30, 30, 64, 2, 3, 1), "conv_fp32_dma "),        # 30 taps: the DMA-staged kernel
    ((2, 3, 30, 30, 18, 3, 3, 1), "conv_fp32_dma "),        # C_o not a multiple of 4
    ((2, 8, 30, 30, 64, 3, 3, 1), "conv_fp32_dma "),        # 16-byte-aligned windows
])
def test_stem32_default(shape, want):
    assert name(shape, "f32").startswith(want)


@pytest.mark.parametrize("shape,want", [
    ((128, 64, 224, 224, 64, 7, 7, 2), "conv_fp32_dma p6c8l8s2k16"),    # K_w > s > 1: the 6-pixel tile
    ((128, 64, 112, 112, 128, 3, 3, 1), "conv_fp32_dma p8c8l8s2k16"),   # stride 1
    ((128, 64, 224, 224, 64, 2, 2, 2), "conv_fp32_dma p8c8l8s2k16"),    # K_w = s: no overlap
    ((2, 16, 23, 41, 40, 7, 7, 2), "conv_fp32_dma p8c8l8s2k16t4"),      # few tiles
    ((128, 512, 14, 14, 512, 3, 3, 1), "conv_fp32_dma p4c8l8s2k16t4w8"),  # 576 tiles: the eight-wave tap split
])
def test_dma32_default(shape, want):
    assert name(shape, "f32") == want


def test_stem32_forced(monkeypatch):
    monkeypatch.setenv("IM2WIN_FP32_KERNEL", "stem")
    assert name((2, 5, 30, 30, 64, 2, 3, 1), "f32") == "conv_fp32_stem k32"
    assert status((2, 3, 30, 30, 64, 5, 5, 1), "f32") == EINVAL    # 75 taps
    assert status((2, 8, 30, 30, 64, 3, 3, 1), "f32") == EINVAL    # aligned windows
    monkeypatch.setenv("IM2WIN_FP32_TILE", "m4n16f")
    assert status((2, 3, 30, 30, 64, 3, 3, 1), "f32") == EINVAL    # two fp32 kernels forced


def test_fp32_column_kernel_forced(monkeypatch):
    monkeypatch.setenv("IM2WIN_FP32_COLS", "k3p256t16")
    assert name((2, 64, 24, 24, 64, 3, 3, 1), "f32") == "conv_fp32_cols k3p256t16"
    assert status((2, 64, 24, 24, 64, 5, 5, 1), "f32") == EINVAL    # a 3-wide variant on a 5x5 layer
    assert status((2, 3, 24, 24, 64, 3, 3, 1), "f32") == EINVAL     # windows not 16-byte aligned
    assert status((2, 512, 7, 7, 512, 3, 3, 1), "f32") == EINVAL    # 52 strip runs: rows past the budget
    monkeypatch.setenv("IM2WIN_FP32_KERNEL", "p8c8l8s2k16")
    assert status((2, 64, 24, 24, 64, 3, 3, 1), "f32") == EINVAL    # two fp32 kernels forced

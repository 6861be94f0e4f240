"""The C-ABI library on the host: it loads, exports every function the header
declares, and its host-only functions and argument checks behave as the header
states.  No call here reaches a GPU."""
import ctypes
import os
import re

import pytest

import paper_2608_20725_amd as pkg
from paper_2608_20725_amd import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "im2win.h")

OK, EINVAL, EALIGN, ERANGE, ENODEV, ELAUNCH, EWORKSPACE, EOVERLAP, EBUFFER = 0, -1, -2, -3, -4, -5, -6, -7, -8


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(pkg.library_path()):
        from paper_2608_20725_amd import build
        build.build()
    return pkg.load_library()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(conv_\w+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ("conv_im2win_transform", "conv_im2win_fp32", "conv_im2win_fp16",
              "conv_workspace_bytes"):
        assert n in names


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_library_exports_nothing_undeclared(lib):
    import subprocess
    out = subprocess.run(["nm", "-D", "--defined-only", pkg.library_path()],
                         capture_output=True, text=True, check=True).stdout
    exported = {l.split()[-1] for l in out.splitlines() if " T " in l}
    ours = {n for n in exported if n.startswith("conv_")}
    assert ours == set(declared_functions())


def _closed_form(l, elt, fp16):
    Ho = (l.H - l.K_h) // l.stride + 1
    Wo = (l.W - l.K_w) // l.stride + 1
    win = l.N * Ho * l.W * l.K_h * l.C_i * elt
    pad_end = (win + 255) // 256 * 256 + 256
    K = l.K_h * l.K_w * l.C_i
    if fp16:   # packed filter round_up(C_o,256) x K_w x round_up(K_h*C_i,64) fp16
        packed = ((l.C_o + 255) // 256 * 256) * l.K_w * ((l.K_h * l.C_i + 63) // 64 * 64) * 2
        assert packed >= ((l.C_o + 255) // 256 * 256) * ((K + 63) // 64 * 64) * 2
    else:      # packed filter: the larger of [round_up(K,16)][round_up(C_o,32)] fp32 (vector-ALU
               # kernels) and round_up(C_o,128) x round_up(K,32) fp32 (matrix-core kernel)
        packed = max(((K + 15) // 16 * 16) * ((l.C_o + 31) // 32 * 32),
                     ((l.C_o + 127) // 128 * 128) * ((K + 31) // 32 * 32)) * 4
    im2col = l.N * Ho * Wo * K * elt
    return pad_end + packed, im2col, win


@pytest.mark.parametrize("layer", workloads.ALL, ids=lambda l: l.name)
def test_workspace_and_im2col_bytes(lib, layer, orc):
    for dt, elt in ((pkg.F32, 4), (pkg.F16, 2), (pkg.BF16, 2)):
        ws, im2col, win = _closed_form(layer, elt, dt != pkg.F32)
        args = (layer.N, layer.C_i, layer.H, layer.W, layer.C_o, layer.K_h, layer.K_w, layer.stride)
        assert pkg.conv_workspace_bytes(*args, dt) == ws
        assert pkg.conv_im2col_bytes(layer.N, layer.C_i, layer.H, layer.W, layer.K_h, layer.K_w,
                                     layer.stride, dt) == im2col
        # the oracle counts the same two tensors from their index ranges
        assert win == elt * orc.window_elems(layer.N, layer.C_i, layer.H, layer.W, layer.K_h,
                                             layer.stride)
        assert im2col == elt * orc.im2col_elems(layer.N, layer.C_i, layer.H, layer.W, layer.K_h,
                                                layer.K_w, layer.stride)
        # the window tensor is smaller than im2col whenever windows overlap
        if layer.K_w > layer.stride:
            assert win < im2col
        else:
            assert win == im2col


def test_output_dims_table1(lib):
    from oracle_checks import read_table
    for row in read_table("table1_layers.txt"):
        _, ci, hi, wi, co, hf, wf, s, oc, ho, wo = map(lambda v: int(v) if v.isdigit() else v, row)
        assert pkg.conv_output_dims(hi, wi, hf, wf, s) == (ho, wo)


@pytest.mark.parametrize("args", [
    (0, 3, 8, 8, 4, 3, 3, 1), (1, 0, 8, 8, 4, 3, 3, 1), (1, 3, 8, 8, 0, 3, 3, 1),
    (1, 3, 8, 8, 4, 9, 3, 1), (1, 3, 8, 8, 4, 3, 9, 1), (1, 3, 8, 8, 4, 3, 3, 0),
    (1, 3, 8, 8, 4, -1, 3, 1), (-2, 3, 8, 8, 4, 3, 3, 1),
])
def test_workspace_rejects_bad_dims(lib, args):
    assert lib.conv_workspace_bytes(*args, pkg.F32) == EINVAL


def test_workspace_rejects_bad_dtype(lib):
    assert lib.conv_workspace_bytes(1, 3, 8, 8, 4, 3, 3, 1, 7) == EINVAL
    assert lib.conv_workspace_bytes(1, 3, 8, 8, 4, 3, 3, 1, 3) == EINVAL
    assert lib.conv_workspace_bytes(1, 3, 8, 8, 4, 3, 3, 1, -1) == EINVAL


def test_ranges(lib):
    # strip W_i*K_h*C_i must stay below 2^20 elements
    assert lib.conv_workspace_bytes(1, 1 << 12, 300, 300, 4, 1, 1, 1, pkg.F32) == ERANGE
    # K_h*K_w*C_i below 2^24
    assert lib.conv_workspace_bytes(1, 1 << 20, 4, 4, 4, 4, 4, 1, pkg.F32) == ERANGE
    # C_o below 2^19
    assert lib.conv_workspace_bytes(1, 3, 8, 8, 1 << 19, 3, 3, 1, pkg.F32) == ERANGE
    # more than 2^31 output pixels
    assert lib.conv_workspace_bytes(1 << 20, 1, 64, 64, 1, 1, 1, 1, pkg.F32) == ERANGE
    # fp16 packed filter of 2^31 bytes or more (fp32 has no such limit)
    assert lib.conv_workspace_bytes(1, 1 << 12, 1, 64, 1 << 16, 1, 64, 1, pkg.F16) == ERANGE
    assert lib.conv_workspace_bytes(1, 1 << 12, 1, 64, 1 << 16, 1, 64, 1, pkg.BF16) == ERANGE
    assert lib.conv_workspace_bytes(1, 1 << 12, 1, 64, 1 << 16, 1, 64, 1, pkg.F32) > 0


def test_output_dims_rejects(lib):
    ho, wo = ctypes.c_int64(), ctypes.c_int64()
    assert lib.conv_output_dims(8, 8, 9, 3, 1, ctypes.byref(ho), ctypes.byref(wo)) == EINVAL
    assert lib.conv_output_dims(8, 8, 3, 3, 0, ctypes.byref(ho), ctypes.byref(wo)) == EINVAL
    assert lib.conv_output_dims(8, 8, 3, 3, 1, None, ctypes.byref(wo)) == EINVAL


def test_null_pointers_rejected_first(lib):
    v = ctypes.c_void_p
    # null pointers win over bad dims
    assert lib.conv_im2win_transform(None, v(256), 1 << 20, 0, 3, 8, 8, 4, 3, 3, 1, 0, None) == EINVAL
    assert lib.conv_im2win_fp32(v(256), 1 << 20, None, v(512), 1, 3, 8, 8, 4, 3, 3, 1, None) == EINVAL
    assert lib.conv_im2win_fp16(v(256), 1 << 20, v(512), None, 1, 3, 8, 8, 4, 3, 3, 1, None) == EINVAL
    assert lib.conv_im2win_bf16(None, 1 << 20, v(512), v(768), 1, 3, 8, 8, 4, 3, 3, 1, None) == EINVAL
    assert lib.conv_im2win_bf16(v(256), 1 << 20, v(512), v(768), 0, 3, 8, 8, 4, 3, 3, 1, None) == EINVAL


def test_misaligned_pointers_rejected(lib):
    v = ctypes.c_void_p
    assert lib.conv_im2win_transform(v(0x1008), v(0x100000), 1 << 20, 1, 3, 8, 8, 4, 3, 3, 1, 0,
                                     None) == EALIGN
    assert lib.conv_im2win_fp32(v(0x100000), 1 << 20, v(0x2004), v(0x3000), 1, 3, 8, 8, 4, 3, 3, 1,
                                None) == EALIGN
    assert lib.conv_im2win_fp16(v(0x100000), 1 << 20, v(0x2000), v(0x3002), 1, 3, 8, 8, 4, 3, 3, 1,
                                None) == EALIGN
    assert lib.conv_im2win_bf16(v(0x100008), 1 << 20, v(0x2000), v(0x3000), 1, 3, 8, 8, 4, 3, 3, 1,
                                None) == EALIGN
    assert lib.conv_im2win_fp32_mfma(v(0x100000), 1 << 20, v(0x2004), v(0x3000), 1, 3, 8, 8, 4, 3, 3, 1,
                                     None) == EALIGN


def test_dims_checked_before_pointers_resolve(lib):
    v = ctypes.c_void_p
    assert lib.conv_im2win_fp32(v(0x100000), 1 << 20, v(0x2000), v(0x3000), 1, 3, 8, 8, 4, 9, 3, 1,
                                None) == EINVAL
    assert lib.conv_im2win_transform(v(0x1000), v(0x100000), 1 << 20, 1, 3, 8, 8, 4, 3, 3, 1, 5,
                                     None) == EINVAL


def test_strerror(lib):
    for code in (OK, EINVAL, EALIGN, ERANGE, ENODEV, ELAUNCH, EWORKSPACE, EOVERLAP, EBUFFER):
        assert pkg.conv_im2win_strerror(code)
    assert pkg.conv_im2win_strerror(12345) == "unknown status"


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    monkeypatch.setattr(pkg, "_lib", None)
    monkeypatch.setattr(pkg, "_LIB_PATH", str(tmp_path / "nope.so"))
    with pytest.raises(RuntimeError, match="not built"):
        pkg.load_library()


@pytest.mark.parametrize("layer", [workloads.CFG2, workloads.CFG3, workloads.CFG4], ids=lambda l: l.name)
def test_chunked_workspace_bytes(lib, layer):
    l = layer
    for dt, elt in ((pkg.F32, 4), (pkg.F16, 2)):
        full, _, _ = _closed_form(l, elt, dt == pkg.F16)
        for n_chunk in (1, 7, l.N, l.N + 5):
            for two in (0, 1):
                nc = min(n_chunk, l.N)
                Ho = (l.H - l.K_h) // l.stride + 1
                win = nc * Ho * l.W * l.K_h * l.C_i * elt
                pad_end = (win + 255) // 256 * 256 + 256
                slot = (pad_end + 255) // 256 * 256
                packed = full - ((l.N * Ho * l.W * l.K_h * l.C_i * elt + 255) // 256 * 256 + 256)
                want = (2 if two else 1) * slot + packed
                got = pkg.conv_chunked_workspace_bytes(l.N, l.C_i, l.H, l.W, l.C_o, l.K_h, l.K_w,
                                                       l.stride, n_chunk, two, dt)
                assert got == want
        # the window-tensor slots of one-image chunks are 2/N of the full batch's
        one = pkg.conv_chunked_workspace_bytes(l.N, l.C_i, l.H, l.W, l.C_o, l.K_h, l.K_w, l.stride,
                                               1, 1, dt)
        assert one - packed < (full - packed) // 16


def test_chunked_rejects(lib):
    assert lib.conv_chunked_workspace_bytes(4, 8, 10, 10, 16, 3, 3, 1, 0, 0, pkg.F32) == EINVAL
    assert lib.conv_chunked_workspace_bytes(4, 8, 10, 10, 16, 3, 3, 1, -3, 1, pkg.F32) == EINVAL
    assert lib.conv_chunked_workspace_bytes(4, 8, 10, 10, 16, 3, 3, 1, 2, 0, 9) == EINVAL
    v = ctypes.c_void_p
    # null pointers first
    assert lib.conv_im2win_chunked(None, v(256), v(512), v(1024), 1 << 20, 4, 8, 10, 10, 16, 3, 3, 1, 2,
                                   pkg.F32, None, None) == EINVAL


def test_padded_transform_checks(lib):
    v = ctypes.c_void_p
    f = lib.conv_im2win_transform_padded
    # null pointers first, then dims: negative pads, a filter larger than the
    # padded input, pads past the range
    assert f(None, v(0x100000), 1 << 20, 1, 3, 8, 8, 4, 3, 3, 1, 1, 1, pkg.F32, None) == EINVAL
    assert f(v(0x1000), v(0x100000), 1 << 20, 1, 3, 8, 8, 4, 3, 3, 1, -1, 0, pkg.F32, None) == EINVAL
    assert f(v(0x1000), v(0x100000), 1 << 20, 1, 3, 8, 8, 4, 3, 3, 1, 0, -2, pkg.F32, None) == EINVAL
    assert f(v(0x1000), v(0x100000), 1 << 20, 1, 3, 2, 2, 4, 5, 5, 1, 1, 1, pkg.F32, None) == EINVAL
    assert f(v(0x1000), v(0x100000), 1 << 20, 1, 3, 8, 8, 4, 3, 3, 1, 1 << 40, 0, pkg.F32, None) == ERANGE
    # a filter that fits only thanks to the padding passes the dims: the
    # misaligned input is what is rejected
    assert f(v(0x1008), v(0x100000), 1 << 20, 1, 3, 2, 2, 4, 3, 3, 1, 1, 1, pkg.F32, None) == EALIGN


@pytest.mark.parametrize("args", [
    # N, C_i, H, W, C_o, K_h, K_w, s, d
    (2, 3, 9, 10, 4, 3, 3, 1, 2), (1, 2, 11, 9, 3, 3, 2, 2, 3), (2, 4, 8, 8, 2, 2, 2, 1, 4),
    (1, 1, 7, 13, 2, 3, 3, 3, 2), (1, 64, 60, 60, 64, 3, 3, 1, 2), (3, 5, 13, 13, 8, 2, 2, 1, 12),
])
def test_dilated_workspace_and_dims(lib, orc, args):
    """The dilated window tensor is the oracle's (residue-grouped strips of
    d*ceil(W/d) columns); workspace = its bytes, the zero pad and the packed
    filter; output extents (H - (K-1)d - 1)/s + 1."""
    import numpy as np
    N, Ci, H, W, Co, Kh, Kw, s, d = args
    for dt, elt in ((pkg.F32, 4), (pkg.F16, 2), (pkg.BF16, 2)):
        win = orc.im2win_dil(np.zeros((N, H, W, Ci), np.float32 if elt == 4 else np.float16), Kh, s, 0, 0, d)
        Ho, Wo = pkg.conv_output_dims_dilated(H, W, Kh, Kw, s, d)
        assert (Ho, Wo) == (orc.dil_extent(H, Kh, s, d), orc.dil_extent(W, Kw, s, d))
        assert win.shape[1] == Ho
        pad_end = (win.nbytes + 255) // 256 * 256 + 256
        K = Kh * Kw * Ci
        if dt == pkg.F32:
            packed = max(((K + 15) // 16 * 16) * ((Co + 31) // 32 * 32), ((Co + 127) // 128 * 128) * ((K + 31) // 32 * 32)) * 4
        else:
            packed = ((Co + 255) // 256 * 256) * Kw * ((Kh * Ci + 63) // 64 * 64) * 2
        assert pkg.conv_workspace_bytes_dilated(N, Ci, H, W, Co, Kh, Kw, s, d, dt) == pad_end + packed
        if d == 1:
            assert pkg.conv_workspace_bytes_dilated(N, Ci, H, W, Co, Kh, Kw, s, 1, dt) == \
                pkg.conv_workspace_bytes(N, Ci, H, W, Co, Kh, Kw, s, dt)


def test_dilated_rejects(lib):
    v = ctypes.c_void_p
    ho, wo = ctypes.c_int64(), ctypes.c_int64()
    # dilation < 1, dilated filter larger than the input
    assert lib.conv_output_dims_dilated(8, 8, 3, 3, 1, 0, ctypes.byref(ho), ctypes.byref(wo)) == EINVAL
    assert lib.conv_output_dims_dilated(8, 8, 3, 3, 1, 4, ctypes.byref(ho), ctypes.byref(wo)) == EINVAL
    assert lib.conv_output_dims_dilated(9, 9, 3, 3, 1, 4, ctypes.byref(ho), ctypes.byref(wo)) == OK
    assert (ho.value, wo.value) == (1, 1)
    assert lib.conv_workspace_bytes_dilated(1, 3, 8, 8, 4, 3, 3, 1, 0, pkg.F32) == EINVAL
    assert lib.conv_workspace_bytes_dilated(1, 3, 8, 8, 4, 3, 3, 1, 4, pkg.F32) == EINVAL
    assert lib.conv_workspace_bytes_dilated(1, 3, 8, 8, 4, 3, 3, 1, 1 << 40, pkg.F32) == ERANGE
    # null pointers first, bad dtype, bad dims before any pointer is resolved
    assert lib.conv_im2win_dilated(None, 1 << 20, v(512), v(768), 1, 3, 8, 8, 4, 3, 3, 1, 2, pkg.F32,
                                   None) == EINVAL
    assert lib.conv_im2win_dilated(v(256), 1 << 20, v(512), v(768), 1, 3, 8, 8, 4, 3, 3, 1, 2, 7, None) == EINVAL
    assert lib.conv_im2win_dilated(v(0x100000), 1 << 20, v(0x2000), v(0x3000), 1, 3, 8, 8, 4, 3, 3, 1, 4,
                                   pkg.F16, None) == EINVAL
    assert lib.conv_im2win_transform_dilated(None, v(256), 1 << 20, 1, 3, 8, 8, 4, 3, 3, 1, 0, 0, 2, 0,
                                             None) == EINVAL
    assert lib.conv_im2win_transform_dilated(v(0x1000), v(0x100000), 1 << 20, 1, 3, 8, 8, 4, 3, 3, 1, 0, 0, 0,
                                             0, None) == EINVAL
    assert lib.conv_im2win_transform_dilated(v(0x1008), v(0x100000), 1 << 20, 1, 3, 8, 8, 4, 3, 3, 1, 1, 1, 2,
                                             0, None) == EALIGN

"""im2win convolution on AMD Instinct MI355X (gfx950).

A thin ctypes binding over ``libim2win.so`` (``include/im2win.h``).  Every
function only marshals arguments: shapes and device pointers of PyTorch
tensors, and the current HIP stream.  All work runs in the library's gfx950
kernels; there is no fallback, and a missing library raises.

    H_o, W_o = conv_output_dims(H_i, W_i, K_h, K_w, stride)
    nbytes   = conv_workspace_bytes(N, C_i, H_i, W_i, C_o, K_h, K_w, stride, dtype)
    conv_im2win_transform(x, ws, C_o, K_h, K_w, stride)        # Sec. III-B, Eq. 2
    conv_im2win_transform_padded(x, ws, C_o, K_h, K_w, stride, pad_h, pad_w)
    conv_im2win_fp32(ws, w, out, N, C_i, H_i, W_i, stride)     # Sec. III-C, Eq. 3
    conv_im2win_fp16(ws, w, out, N, C_i, H_i, W_i, stride)     # Sec. III-D, Alg. 1
    conv_im2win_bf16(ws, w, out, N, C_i, H_i, W_i, stride)     # same, bf16 operands
    conv_im2win_fp32_mfma(ws, w, out, N, C_i, H_i, W_i, stride)  # fp32 on the matrix cores
    conv_im2win_transform_dilated(x, ws, C_o, K_h, K_w, stride, pad_h, pad_w, dilation)
    conv_im2win_dilated(ws, w, out, N, C_i, H_p, W_p, stride, dilation)

Layouts: ``x`` NHWC, ``w`` [K_h][K_w][C_i][C_o], ``out`` NHWC; ``ws`` is a
flat byte tensor on the same device.
"""
from __future__ import annotations

import ctypes
import os

__all__ = [
    "Im2winError", "load_library", "library_path", "F32", "F16", "BF16",
    "conv_output_dims", "conv_workspace_bytes", "conv_im2col_bytes",
    "conv_im2win_transform", "conv_im2win_transform_padded", "conv_im2win_fp32", "conv_im2win_fp16",
    "conv_im2win_bf16", "conv_im2win_fp32_mfma", "conv_output_dims_dilated", "conv_workspace_bytes_dilated",
    "conv_im2win_transform_dilated", "conv_im2win_dilated",
    "conv_im2win_strerror", "conv_im2win_kernel_name", "im2win_conv2d",
]

F32 = 0
F16 = 1
BF16 = 2

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libim2win.so")
_lib = None

_i64 = ctypes.c_int64
_vp = ctypes.c_void_p


class Im2winError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__("%s: %s (status %d)" % (what, conv_im2win_strerror(status), status))


def library_path() -> str:
    return _LIB_PATH


def load_library():
    """Loads libim2win.so from the package directory (built in-tree)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise RuntimeError("libim2win.so is not built (expected at %s); run "
                           "`python -c 'import __graft_entry__ as g; g.build()'`" % _LIB_PATH)
    lib = ctypes.CDLL(_LIB_PATH)
    lib.conv_output_dims.restype = ctypes.c_int
    lib.conv_output_dims.argtypes = [_i64] * 5 + [ctypes.POINTER(_i64)] * 2
    lib.conv_workspace_bytes.restype = _i64
    lib.conv_workspace_bytes.argtypes = [_i64] * 8 + [ctypes.c_int]
    lib.conv_im2col_bytes.restype = _i64
    lib.conv_im2col_bytes.argtypes = [_i64] * 7 + [ctypes.c_int]
    lib.conv_im2win_transform.restype = ctypes.c_int
    lib.conv_im2win_transform.argtypes = [_vp, _vp, _i64] + [_i64] * 8 + [ctypes.c_int, _vp]
    lib.conv_im2win_transform_padded.restype = ctypes.c_int
    lib.conv_im2win_transform_padded.argtypes = [_vp, _vp, _i64] + [_i64] * 10 + [ctypes.c_int, _vp]
    lib.conv_im2win_fp32.restype = ctypes.c_int
    lib.conv_im2win_fp32.argtypes = [_vp, _i64, _vp, _vp] + [_i64] * 8 + [_vp]
    lib.conv_im2win_fp16.restype = ctypes.c_int
    lib.conv_im2win_fp16.argtypes = [_vp, _i64, _vp, _vp] + [_i64] * 8 + [_vp]
    lib.conv_im2win_bf16.restype = ctypes.c_int
    lib.conv_im2win_bf16.argtypes = [_vp, _i64, _vp, _vp] + [_i64] * 8 + [_vp]
    lib.conv_im2win_fp32_mfma.restype = ctypes.c_int
    lib.conv_im2win_fp32_mfma.argtypes = [_vp, _i64, _vp, _vp] + [_i64] * 8 + [_vp]
    lib.conv_output_dims_dilated.restype = ctypes.c_int
    lib.conv_output_dims_dilated.argtypes = [_i64] * 6 + [ctypes.POINTER(_i64)] * 2
    lib.conv_workspace_bytes_dilated.restype = _i64
    lib.conv_workspace_bytes_dilated.argtypes = [_i64] * 9 + [ctypes.c_int]
    lib.conv_im2win_transform_dilated.restype = ctypes.c_int
    lib.conv_im2win_transform_dilated.argtypes = [_vp, _vp, _i64] + [_i64] * 11 + [ctypes.c_int, _vp]
    lib.conv_im2win_dilated.restype = ctypes.c_int
    lib.conv_im2win_dilated.argtypes = [_vp, _i64, _vp, _vp] + [_i64] * 9 + [ctypes.c_int, _vp]
    lib.conv_chunked_workspace_bytes.restype = _i64
    lib.conv_chunked_workspace_bytes.argtypes = [_i64] * 9 + [ctypes.c_int, ctypes.c_int]
    lib.conv_im2win_chunked.restype = ctypes.c_int
    lib.conv_im2win_chunked.argtypes = [_vp, _vp, _vp, _vp, _i64] + [_i64] * 9 + [ctypes.c_int, _vp, _vp]
    lib.conv_im2win_kernel_name.restype = ctypes.c_int
    lib.conv_im2win_kernel_name.argtypes = [_i64] * 9 + [ctypes.c_int, ctypes.c_int, ctypes.c_char_p, _i64]
    lib.conv_im2win_strerror.restype = ctypes.c_char_p
    lib.conv_im2win_strerror.argtypes = [ctypes.c_int]
    _lib = lib
    return lib


def conv_im2win_strerror(status: int) -> str:
    return load_library().conv_im2win_strerror(int(status)).decode()


def _dtype_code(dtype) -> int:
    import torch
    if dtype in (F32, "f32", "fp32", torch.float32):
        return F32
    if dtype in (F16, "f16", "fp16", torch.float16):
        return F16
    if dtype in (BF16, "bf16", torch.bfloat16):
        return BF16
    raise ValueError("dtype must be fp32, fp16 or bf16, got %r" % (dtype,))


def _stream(stream):
    import torch
    if stream is None:
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return ctypes.c_void_p(stream)
    return ctypes.c_void_p(stream.cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr())


def _nbytes(t) -> int:
    return t.numel() * t.element_size()


def _check(rc: int, what: str):
    if rc != 0:
        raise Im2winError(rc, what)


def conv_im2win_kernel_name(N, C_i, H_i, W_i, C_o, K_h, K_w, stride, dtype, dilation: int = 1,
                            fp32_matrix_cores: bool = False) -> str:
    """The kernel (family and variant) the conv call of this layer runs."""
    buf = ctypes.create_string_buffer(64)
    _check(load_library().conv_im2win_kernel_name(N, C_i, H_i, W_i, C_o, K_h, K_w, stride, dilation,
                                                  _dtype_code(dtype), 1 if fp32_matrix_cores else 0,
                                                  buf, len(buf)), "conv_im2win_kernel_name")
    return buf.value.decode()


def conv_output_dims(H_i: int, W_i: int, K_h: int, K_w: int, stride: int):
    ho, wo = _i64(), _i64()
    _check(load_library().conv_output_dims(H_i, W_i, K_h, K_w, stride,
                                           ctypes.byref(ho), ctypes.byref(wo)), "conv_output_dims")
    return ho.value, wo.value


def conv_workspace_bytes(N, C_i, H_i, W_i, C_o, K_h, K_w, stride, dtype) -> int:
    n = load_library().conv_workspace_bytes(N, C_i, H_i, W_i, C_o, K_h, K_w, stride,
                                            _dtype_code(dtype))
    if n < 0:
        raise Im2winError(int(n), "conv_workspace_bytes")
    return int(n)


def conv_im2col_bytes(N, C_i, H_i, W_i, K_h, K_w, stride, dtype) -> int:
    n = load_library().conv_im2col_bytes(N, C_i, H_i, W_i, K_h, K_w, stride, _dtype_code(dtype))
    if n < 0:
        raise Im2winError(int(n), "conv_im2col_bytes")
    return int(n)


def conv_im2win_transform(x, ws, C_o: int, K_h: int, K_w: int, stride: int, stream=None):
    """Writes the window tensor of NHWC input ``x`` (fp32, fp16 or bf16) into ``ws``."""
    if x.dim() != 4 or not x.is_contiguous():
        raise ValueError("x must be a contiguous NHWC tensor")
    N, H_i, W_i, C_i = x.shape
    rc = load_library().conv_im2win_transform(
        _ptr(x), _ptr(ws), _nbytes(ws), N, C_i, H_i, W_i, C_o, K_h, K_w, stride,
        _dtype_code(x.dtype), _stream(stream))
    _check(rc, "conv_im2win_transform")


def conv_im2win_transform_padded(x, ws, C_o: int, K_h: int, K_w: int, stride: int, pad_h: int,
                                 pad_w: int, stream=None):
    """Writes the window tensor of ``x`` zero-padded by ``pad_h`` rows and
    ``pad_w`` columns on each side into ``ws`` (sized for the padded extents);
    the convolutions then take ``H_i + 2*pad_h`` and ``W_i + 2*pad_w``."""
    if x.dim() != 4 or not x.is_contiguous():
        raise ValueError("x must be a contiguous NHWC tensor")
    N, H_i, W_i, C_i = x.shape
    rc = load_library().conv_im2win_transform_padded(
        _ptr(x), _ptr(ws), _nbytes(ws), N, C_i, H_i, W_i, C_o, K_h, K_w, stride, pad_h, pad_w,
        _dtype_code(x.dtype), _stream(stream))
    _check(rc, "conv_im2win_transform_padded")


def _conv(fn, what, ws, w, out, N, C_i, H_i, W_i, stride, stream):
    if w.dim() != 4 or not w.is_contiguous() or not out.is_contiguous():
        raise ValueError("w must be a contiguous [K_h][K_w][C_i][C_o] tensor, out contiguous")
    K_h, K_w, C_i2, C_o = w.shape
    if C_i2 != C_i:
        raise ValueError("filter has %d input channels, layer has %d" % (C_i2, C_i))
    rc = fn(_ptr(ws), _nbytes(ws), _ptr(w), _ptr(out), N, C_i, H_i, W_i, C_o, K_h, K_w, stride,
            _stream(stream))
    _check(rc, what)


def conv_im2win_fp32(ws, w, out, N: int, C_i: int, H_i: int, W_i: int, stride: int, stream=None):
    """fp32 conv from the fp32 window tensor in ``ws``; ``out`` is NHWC fp32."""
    import torch
    if w.dtype != torch.float32 or out.dtype != torch.float32:
        raise TypeError("conv_im2win_fp32 takes fp32 filter and output")
    _conv(load_library().conv_im2win_fp32, "conv_im2win_fp32", ws, w, out, N, C_i, H_i, W_i,
          stride, stream)


def conv_im2win_fp16(ws, w, out, N: int, C_i: int, H_i: int, W_i: int, stride: int, stream=None):
    """fp16 conv (fp32 accumulation) from the fp16 window tensor in ``ws``."""
    import torch
    if w.dtype != torch.float16 or out.dtype != torch.float16:
        raise TypeError("conv_im2win_fp16 takes fp16 filter and output")
    _conv(load_library().conv_im2win_fp16, "conv_im2win_fp16", ws, w, out, N, C_i, H_i, W_i,
          stride, stream)


def conv_im2win_bf16(ws, w, out, N: int, C_i: int, H_i: int, W_i: int, stride: int, stream=None):
    """bf16 conv (fp32 accumulation) from the bf16 window tensor in ``ws``."""
    import torch
    if w.dtype != torch.bfloat16 or out.dtype != torch.bfloat16:
        raise TypeError("conv_im2win_bf16 takes bf16 filter and output")
    _conv(load_library().conv_im2win_bf16, "conv_im2win_bf16", ws, w, out, N, C_i, H_i, W_i,
          stride, stream)


def conv_im2win_fp32_mfma(ws, w, out, N: int, C_i: int, H_i: int, W_i: int, stride: int, stream=None):
    """fp32 conv on the matrix cores (an alternate fp32 path) from the fp32
    window tensor in ``ws``; layers with C_i not a multiple of 4 run on the
    vector ALUs."""
    import torch
    if w.dtype != torch.float32 or out.dtype != torch.float32:
        raise TypeError("conv_im2win_fp32_mfma takes fp32 filter and output")
    _conv(load_library().conv_im2win_fp32_mfma, "conv_im2win_fp32_mfma", ws, w, out, N, C_i, H_i, W_i,
          stride, stream)


def conv_for_dtype(dtype):
    """The conv entry point for an element type (fp32, fp16 or bf16)."""
    return (conv_im2win_fp32, conv_im2win_fp16, conv_im2win_bf16)[_dtype_code(dtype)]


def im2win_conv2d(x, w, stride: int, ws=None, out=None, stream=None):
    """Transform + conv on the current stream; allocates what is not given.

    Returns (out, ws)."""
    import torch
    N, H_i, W_i, C_i = x.shape
    K_h, K_w, _, C_o = w.shape
    H_o, W_o = conv_output_dims(H_i, W_i, K_h, K_w, stride)
    need = conv_workspace_bytes(N, C_i, H_i, W_i, C_o, K_h, K_w, stride, x.dtype)
    if ws is None:
        ws = torch.empty(need, dtype=torch.uint8, device=x.device)
    if out is None:
        out = torch.empty((N, H_o, W_o, C_o), dtype=x.dtype, device=x.device)
    conv_im2win_transform(x, ws, C_o, K_h, K_w, stride, stream)
    conv_for_dtype(x.dtype)(ws, w, out, N, C_i, H_i, W_i, stride, stream)
    return out, ws


def conv_chunked_workspace_bytes(N, C_i, H_i, W_i, C_o, K_h, K_w, stride, n_chunk, two_streams,
                                 dtype) -> int:
    n = load_library().conv_chunked_workspace_bytes(N, C_i, H_i, W_i, C_o, K_h, K_w, stride, n_chunk,
                                                    1 if two_streams else 0, _dtype_code(dtype))
    if n < 0:
        raise Im2winError(int(n), "conv_chunked_workspace_bytes")
    return int(n)


def conv_im2win_chunked(x, w, out, ws, stride: int, n_chunk: int, stream=None, aux_stream=None):
    """Transform + conv of NHWC ``x`` in chunks of ``n_chunk`` images into
    ``out``; with ``aux_stream`` the transform of the next chunk overlaps the
    conv of the current one."""
    import torch
    if x.dim() != 4 or not x.is_contiguous() or w.dim() != 4 or not w.is_contiguous():
        raise ValueError("x must be contiguous NHWC, w contiguous [K_h][K_w][C_i][C_o]")
    if not out.is_contiguous() or x.dtype != w.dtype or x.dtype != out.dtype:
        raise ValueError("out must be contiguous, with the dtype of x and w")
    N, H_i, W_i, C_i = x.shape
    K_h, K_w, C_i2, C_o = w.shape
    if C_i2 != C_i:
        raise ValueError("filter has %d input channels, layer has %d" % (C_i2, C_i))
    aux = ctypes.c_void_p(None) if aux_stream is None else _stream(aux_stream)
    rc = load_library().conv_im2win_chunked(
        _ptr(x), _ptr(w), _ptr(out), _ptr(ws), _nbytes(ws), N, C_i, H_i, W_i, C_o, K_h, K_w,
        stride, n_chunk, _dtype_code(x.dtype), _stream(stream), aux)
    _check(rc, "conv_im2win_chunked")



def conv_output_dims_dilated(H_i: int, W_i: int, K_h: int, K_w: int, stride: int, dilation: int):
    ho, wo = _i64(), _i64()
    _check(load_library().conv_output_dims_dilated(H_i, W_i, K_h, K_w, stride, dilation,
                                                   ctypes.byref(ho), ctypes.byref(wo)),
           "conv_output_dims_dilated")
    return ho.value, wo.value


def conv_workspace_bytes_dilated(N, C_i, H_i, W_i, C_o, K_h, K_w, stride, dilation, dtype) -> int:
    n = load_library().conv_workspace_bytes_dilated(N, C_i, H_i, W_i, C_o, K_h, K_w, stride, dilation,
                                                    _dtype_code(dtype))
    if n < 0:
        raise Im2winError(int(n), "conv_workspace_bytes_dilated")
    return int(n)


def conv_im2win_transform_dilated(x, ws, C_o: int, K_h: int, K_w: int, stride: int, pad_h: int, pad_w: int,
                                  dilation: int, stream=None):
    """Writes the dilated window tensor of ``x`` zero-padded by ``pad_h`` /
    ``pad_w`` into ``ws`` (sized by conv_workspace_bytes_dilated for the
    padded extents)."""
    if x.dim() != 4 or not x.is_contiguous():
        raise ValueError("x must be a contiguous NHWC tensor")
    N, H_i, W_i, C_i = x.shape
    rc = load_library().conv_im2win_transform_dilated(
        _ptr(x), _ptr(ws), _nbytes(ws), N, C_i, H_i, W_i, C_o, K_h, K_w, stride, pad_h, pad_w, dilation,
        _dtype_code(x.dtype), _stream(stream))
    _check(rc, "conv_im2win_transform_dilated")


def conv_im2win_dilated(ws, w, out, N: int, C_i: int, H_i: int, W_i: int, stride: int, dilation: int,
                        stream=None):
    """Dilated conv from the dilated window tensor in ``ws``; the precision
    follows ``w`` (fp32 on the vector ALUs, fp16 / bf16 on the matrix cores);
    ``H_i``, ``W_i`` are the padded extents the window tensor was built for."""
    if w.dim() != 4 or not w.is_contiguous() or not out.is_contiguous() or out.dtype != w.dtype:
        raise ValueError("w must be a contiguous [K_h][K_w][C_i][C_o] tensor, out contiguous of w's dtype")
    K_h, K_w, C_i2, C_o = w.shape
    if C_i2 != C_i:
        raise ValueError("filter has %d input channels, layer has %d" % (C_i2, C_i))
    rc = load_library().conv_im2win_dilated(_ptr(ws), _nbytes(ws), _ptr(w), _ptr(out), N, C_i, H_i, W_i, C_o,
                                            K_h, K_w, stride, dilation, _dtype_code(w.dtype), _stream(stream))
    _check(rc, "conv_im2win_dilated")

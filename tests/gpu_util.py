"""Helpers of the GPU parity tests: run the C-ABI path with poisoned outputs
and guard bands, and compare with the fp64 oracle."""
from __future__ import annotations

import numpy as np
import torch

import oracle
import paper_2608_20725_amd as pkg

GUARD = 256            # elements of guard band on each side of an output
WS_GUARD = 4096        # bytes of sentinel after the workspace
SENTINEL = 0xA5

# bf16: one output rounding costs at most 2^-8 |y| <= 2^-8 sum|x||w| (8-bit
# significand, nearest-even), fp32 accumulation at most K 2^-24 sum|x||w|
# <= 2.8e-4 for the K <= 4608 tested here: 3.91e-3 + 0.28e-3 < 4.5e-3.
TOL = {torch.float32: 1e-5, torch.float16: 2e-3, torch.bfloat16: 4.5e-3}


def say(*a):
    print(*a, flush=True)


class Run:
    """One transform + conv through the C ABI, on `stream` (default: current)."""

    def __init__(self, x, w, stride, dtype, stream=None, conv=True):
        dev = torch.device("cuda")
        self.N, self.H, self.W, self.Ci = x.shape
        self.Kh, self.Kw, _, self.Co = w.shape
        self.s = stride
        self.dtype = dtype
        self.Ho, self.Wo = pkg.conv_output_dims(self.H, self.W, self.Kh, self.Kw, stride)
        self.need = pkg.conv_workspace_bytes(self.N, self.Ci, self.H, self.W, self.Co, self.Kh,
                                             self.Kw, stride, dtype)
        self.xd = x.to(dtype).contiguous().to(dev)
        self.wd = w.to(dtype).contiguous().to(dev)
        self.ws_all = torch.full((self.need + WS_GUARD,), SENTINEL, dtype=torch.uint8, device=dev)
        self.ws = self.ws_all[:self.need]
        n_out = self.N * self.Ho * self.Wo * self.Co
        self.out_all = torch.full((GUARD + n_out + GUARD,), float("nan"), dtype=dtype, device=dev)
        self.out = self.out_all[GUARD:GUARD + n_out].view(self.N, self.Ho, self.Wo, self.Co)
        pkg.conv_im2win_transform(self.xd, self.ws, self.Co, self.Kh, self.Kw, stride, stream)
        if conv:
            pkg.conv_for_dtype(dtype)(self.ws, self.wd, self.out, self.N, self.Ci, self.H, self.W, stride, stream)
        torch.cuda.synchronize()

    def rerun_conv(self):
        pkg.conv_for_dtype(self.dtype)(self.ws, self.wd, self.out, self.N, self.Ci, self.H, self.W, self.s)
        torch.cuda.synchronize()

    def window_bytes(self):
        return self.N * self.Ho * self.W * self.Kh * self.Ci * self.xd.element_size()

    def check_workspace_guard(self):
        tail = self.ws_all[self.need:].cpu().numpy()
        assert np.all(tail == SENTINEL), "bytes written past the workspace"

    def check_out_guards(self):
        g = self.out_all.cpu()
        assert torch.isnan(g[:GUARD].float()).all(), "write before the output"
        assert torch.isnan(g[-GUARD:].float()).all(), "write past the output"

    def out_np(self):
        return self.out.float().cpu().numpy().astype(np.float64)


def rel_err(y, ref, absref):
    """max |y - ref| / sum|x||w|; where the sum is 0, y must be exactly 0."""
    y = np.asarray(y, np.float64)
    zero = absref == 0
    assert np.all(y[zero] == 0), "nonzero output where every product is zero"
    if not np.any(~zero):
        return 0.0
    return float(np.max(np.abs(y[~zero] - ref[~zero]) / absref[~zero]))


def oracle_inputs(x, w, dtype):
    """fp64 copies of the inputs as the path sees them (fp16, bf16: rounded first)."""
    return x.to(dtype).double().numpy(), w.to(dtype).double().numpy()


def check_full(run, x, w):
    """Every output against the oracle."""
    xo, wo = oracle_inputs(x, w, run.dtype)
    ref, absref = oracle.conv(xo, wo, run.s, with_abs=True)
    y = run.out_np()
    assert not np.isnan(y).any(), "output element left unwritten"
    r = rel_err(y, ref, absref)
    assert r <= TOL[run.dtype], "max |err|/sum|x||w| = %.3g" % r
    return r


def sample_points(N, Ho, Wo, Co, seed, full_images=(0, -1), n_random=4096, max_mac=None, K=None):
    """All outputs of the listed images (as many as `max_mac` multiply-adds
    allow, at least the first) plus `n_random` seeded random outputs."""
    rng = np.random.default_rng(seed)
    pts = []
    imgs = sorted({i % N for i in full_images})
    if max_mac is not None and K is not None:
        # as many of the listed images as the MAC budget allows, at least one
        per = Ho * Wo * Co * K
        imgs = imgs[:max(1, int(max_mac // per))]
    for i in imgs:
        g = np.stack(np.meshgrid([i], np.arange(Ho), np.arange(Wo), np.arange(Co),
                                 indexing="ij"), -1).reshape(-1, 4)
        pts.append(g)
    r = np.stack([rng.integers(0, N, n_random), rng.integers(0, Ho, n_random),
                  rng.integers(0, Wo, n_random), rng.integers(0, Co, n_random)], -1)
    pts.append(r)
    return np.concatenate(pts).astype(np.int64)


def check_sampled(run, x, w, seed=0, max_mac=6e9):
    """Outputs of images 0 and N-1 plus random outputs, each against the
    oracle computed one by one (only the images they touch go to the oracle)."""
    K = run.Kh * run.Kw * run.Ci
    pts = sample_points(run.N, run.Ho, run.Wo, run.Co, seed, max_mac=max_mac, K=K)
    imgs = np.unique(pts[:, 0])
    remap = {int(i): k for k, i in enumerate(imgs)}
    xs = x[torch.from_numpy(imgs)]
    xo, wo = oracle_inputs(xs, w, run.dtype)
    local = pts.copy()
    local[:, 0] = [remap[int(i)] for i in pts[:, 0]]
    ref, absref = oracle.conv_points(xo, wo, run.s, local)
    y = run.out.float().cpu().numpy()
    assert not np.isnan(y).any(), "output element left unwritten"
    got = y[pts[:, 0], pts[:, 1], pts[:, 2], pts[:, 3]].astype(np.float64)
    r = rel_err(got, ref, absref)
    assert r <= TOL[run.dtype], "max |err|/sum|x||w| = %.3g on %d sampled outputs" % (r, len(pts))
    return r, len(pts)


FAMILY = {"pipe": "conv_fp16_pipe", "regs": None}


def assert_kernel(shape, dtype, var, value, dilation=1):
    """The library reports that the forced kernel is the one the call runs."""
    N, Ci, H, W, Co, Kh, Kw, s = shape
    got = pkg.conv_im2win_kernel_name(N, Ci, H, W, Co, Kh, Kw, s, dtype, dilation=dilation)
    if value == "regs":
        want = "conv_fp32_kernel" if var.startswith("IM2WIN_FP32") else "conv_fp16_kernel"
        assert got.split()[0] == want, got
    elif value == "pipe":
        assert got.split()[0] == "conv_fp16_pipe", got
    elif value == "stem":
        want = "conv_fp32_stem" if var.startswith("IM2WIN_FP32") else "conv_fp16_stem"
        assert got.split()[0] == want, got
    else:
        assert got.split()[1] == value, got
    return got

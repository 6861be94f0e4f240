"""Pins of the fp64 oracle against facts that do not come from the oracle.

Each check takes an oracle module (the real one, or a copy with a planted
mistake) and raises AssertionError when the oracle disagrees with:
  * the output sizes printed in the paper (Table I, Fig. 1 caption);
  * an independent library routine (torch ``conv2d`` in fp64 on the CPU, a
    numpy matmul, numpy strided slicing);
  * closed forms and special cases (1x1 conv, delta filter, full-size filter,
    window-tensor and im2col sizes);
  * invariants (linearity, the |x||w| sum, Eq. 3 == Eq. 1).
The checks are sized to run in well under a second each.
"""
from __future__ import annotations

import os

import numpy as np
import torch

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def read_table(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                rows.append(line.split())
    return rows


def _rng(seed):
    return np.random.default_rng(seed)


def _torch_conv(x, w, s):
    """torch conv2d in fp64 on the CPU; NHWC / KhKwCiCo in and out."""
    xt = torch.from_numpy(np.ascontiguousarray(x, np.float64)).permute(0, 3, 1, 2)
    wt = torch.from_numpy(np.ascontiguousarray(w, np.float64)).permute(3, 2, 0, 1)
    y = torch.nn.functional.conv2d(xt, wt.contiguous(), stride=s)
    return y.permute(0, 2, 3, 1).contiguous().numpy()


def _slice_conv(x, w, s):
    """sum over taps of strided input slices times the tap's C_i x C_o matrix."""
    N, H, W, Ci = x.shape
    Kh, Kw, _, Co = w.shape
    Ho, Wo = (H - Kh) // s + 1, (W - Kw) // s + 1
    out = np.zeros((N, Ho, Wo, Co), dtype=np.result_type(x, w))
    for u in range(Kh):
        for v in range(Kw):
            patch = x[:, u:u + s * (Ho - 1) + 1:s, v:v + s * (Wo - 1) + 1:s, :]
            out += patch @ w[u, v]
    return out


# Tiny shapes with K_h != K_w, strides 1..3, ragged sizes.
TINY = [
    # N, Ci, H, W, Co, Kh, Kw, s
    (1, 1, 3, 3, 1, 2, 2, 1),
    (2, 3, 7, 9, 4, 3, 2, 1),
    (1, 4, 9, 8, 3, 2, 4, 2),
    (2, 2, 8, 9, 2, 4, 3, 3),
    (1, 3, 5, 6, 5, 1, 3, 2),
    (2, 4, 6, 5, 3, 3, 1, 1),
]


def check_table1_extents(orc):
    for row in read_table("table1_layers.txt"):
        _, ci, hi, wi, co, hf, wf, s, oc, ho, wo = row
        ci, hi, wi, co, hf, wf, s, oc, ho, wo = map(int, (ci, hi, wi, co, hf, wf, s, oc, ho, wo))
        assert orc.out_extent(hi, hf, s) == ho, row
        assert orc.out_extent(wi, wf, s) == wo, row
        assert oc == co


def check_fig1_shapes(orc):
    for row in read_table("fig1_shapes.txt"):
        n, ci, hi, wi, co, hf, wf, s, ho, wo = map(int, row)
        x = np.ones((n, hi, wi, ci))
        w = np.ones((hf, wf, ci, co))
        y = orc.conv(x, w, s)
        assert y.shape == (n, ho, wo, co)
        # all-ones: every output is the window size
        assert np.all(y == hf * wf * ci)


def check_vs_torch_conv2d(orc):
    for t, (N, Ci, H, W, Co, Kh, Kw, s) in enumerate(TINY):
        r = _rng(10 + t)
        x = r.uniform(-1, 1, (N, H, W, Ci))
        w = r.uniform(-1, 1, (Kh, Kw, Ci, Co))
        y = orc.conv(x, w, s)
        ref = _torch_conv(x, w, s)
        assert y.shape == ref.shape, (y.shape, ref.shape)
        np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)


def check_vs_strided_slices(orc):
    for t, (N, Ci, H, W, Co, Kh, Kw, s) in enumerate(TINY):
        r = _rng(20 + t)
        x = r.integers(-2, 3, (N, H, W, Ci)).astype(np.int64)
        w = r.integers(-2, 3, (Kh, Kw, Ci, Co)).astype(np.int64)
        y = orc.conv(x, w, s)
        ref = _slice_conv(x, w, s)          # exact integer arithmetic
        assert y.shape == ref.shape
        assert np.array_equal(y, ref.astype(np.float64))


def check_1x1_is_matmul(orc):
    r = _rng(3)
    x = r.uniform(-1, 1, (2, 5, 4, 6))
    w = r.uniform(-1, 1, (1, 1, 6, 7))
    y = orc.conv(x, w, 1)
    ref = (x.reshape(-1, 6) @ w.reshape(6, 7)).reshape(2, 5, 4, 7)
    np.testing.assert_allclose(y, ref, rtol=1e-13, atol=1e-13)


def check_delta_filter(orc):
    # F[u0][v0][r][j] = (r == j): the output is a shifted, strided copy
    for (N, Ci, H, W, Kh, Kw, s, u0, v0) in [(2, 3, 9, 8, 3, 2, 2, 2, 1),
                                             (1, 4, 7, 7, 2, 3, 3, 1, 2)]:
        r = _rng(4)
        x = r.uniform(-1, 1, (N, H, W, Ci))
        w = np.zeros((Kh, Kw, Ci, Ci))
        for c in range(Ci):
            w[u0, v0, c, c] = 1.0
        y = orc.conv(x, w, s)
        Ho, Wo = y.shape[1], y.shape[2]
        for m in range(Ho):
            for n in range(Wo):
                assert np.array_equal(y[:, m, n, :], x[:, m * s + u0, n * s + v0, :])


def check_full_filter_is_dot(orc):
    r = _rng(5)
    x = r.uniform(-1, 1, (3, 4, 5, 2))
    w = r.uniform(-1, 1, (4, 5, 2, 3))
    y = orc.conv(x, w, 2)
    assert y.shape == (3, 1, 1, 3)
    ref = np.tensordot(x, w, axes=([1, 2, 3], [0, 1, 2]))
    np.testing.assert_allclose(y[:, 0, 0, :], ref, rtol=1e-13, atol=1e-13)


def check_linearity(orc):
    r = _rng(6)
    N, Ci, H, W, Co, Kh, Kw, s = TINY[2]
    x1, x2 = r.uniform(-1, 1, (2, N, H, W, Ci))
    w1, w2 = r.uniform(-1, 1, (2, Kh, Kw, Ci, Co))
    a, b = 0.75, -1.25          # exact binary fractions
    np.testing.assert_allclose(orc.conv(a * x1 + b * x2, w1, s),
                               a * orc.conv(x1, w1, s) + b * orc.conv(x2, w1, s),
                               rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(orc.conv(x1, a * w1 + b * w2, s),
                               a * orc.conv(x1, w1, s) + b * orc.conv(x1, w2, s),
                               rtol=1e-12, atol=1e-12)


def check_abs_sum(orc):
    # A = sum |x||w| equals the convolution of |x| with |w|, and bounds |O|
    for t, (N, Ci, H, W, Co, Kh, Kw, s) in enumerate(TINY):
        r = _rng(30 + t)
        x = r.uniform(-1, 1, (N, H, W, Ci))
        w = r.uniform(-1, 1, (Kh, Kw, Ci, Co))
        y, a = orc.conv(x, w, s, with_abs=True)
        np.testing.assert_allclose(a, _torch_conv(np.abs(x), np.abs(w), s), rtol=1e-12, atol=1e-12)
        assert np.all(np.abs(y) <= a * (1 + 1e-12))


def check_points(orc):
    N, Ci, H, W, Co, Kh, Kw, s = TINY[3]
    r = _rng(7)
    x = r.uniform(-1, 1, (N, H, W, Ci))
    w = r.uniform(-1, 1, (Kh, Kw, Ci, Co))
    y, a = orc.conv(x, w, s, with_abs=True)
    idx = np.stack(np.meshgrid(*[np.arange(d) for d in y.shape], indexing="ij"), -1).reshape(-1, 4)
    yp, ap = orc.conv_points(x, w, s, idx)
    assert np.array_equal(yp, y.reshape(-1))
    assert np.array_equal(ap, a.reshape(-1))


def _numpy_im2win(x, Kh, s):
    """Eq. (2) built from array slicing: strip m stacks input rows m*s..m*s+Kh-1
    column by column."""
    N, H, W, Ci = x.shape
    Ho = (H - Kh) // s + 1
    rows = np.stack([x[:, m * s:m * s + Kh] for m in range(Ho)], axis=1)   # N,Ho,Kh,W,Ci
    return np.ascontiguousarray(rows.transpose(0, 1, 3, 2, 4)).reshape(N, Ho, W * Kh, Ci)


def check_im2win_layout(orc):
    for t, (N, Ci, H, W, Co, Kh, Kw, s) in enumerate(TINY):
        r = _rng(40 + t)
        for dt in (np.float32, np.float16):
            x = r.uniform(-1, 1, (N, H, W, Ci)).astype(dt)
            win = orc.im2win(x, Kh, s)
            assert win.dtype == dt
            assert win.tobytes() == _numpy_im2win(x, Kh, s).tobytes()


def check_im2win_identity(orc):
    # K_h = 1, s = 1: Eq. (2) reduces to the identity
    r = _rng(8)
    x = r.uniform(-1, 1, (2, 5, 7, 3)).astype(np.float32)
    assert orc.im2win(x, 1, 1).tobytes() == x.tobytes()


def check_windows_contiguous(orc):
    # each output's window is one contiguous span of its strip, ordered
    # (filter column, filter row, channel)
    for t, (N, Ci, H, W, Co, Kh, Kw, s) in enumerate(TINY):
        r = _rng(50 + t)
        x = r.uniform(-1, 1, (N, H, W, Ci)).astype(np.float32)
        win = orc.im2win(x, Kh, s).reshape(N, -1, W * Kh * Ci)
        Ho, Wo = (H - Kh) // s + 1, (W - Kw) // s + 1
        K = Kh * Kw * Ci
        for i in range(N):
            for m in range(Ho):
                for n in range(Wo):
                    span = win[i, m, n * s * Kh * Ci: n * s * Kh * Ci + K]
                    patch = x[i, m * s:m * s + Kh, n * s:n * s + Kw, :]     # u, v, r
                    assert np.array_equal(span, patch.transpose(1, 0, 2).reshape(-1))


def check_windowed_equals_direct(orc):
    for t, (N, Ci, H, W, Co, Kh, Kw, s) in enumerate(TINY):
        r = _rng(60 + t)
        x = r.uniform(-1, 1, (N, H, W, Ci))
        w = r.uniform(-1, 1, (Kh, Kw, Ci, Co))
        win = orc.im2win(x, Kh, s)
        np.testing.assert_allclose(orc.windowed_conv(win, w, H, W, s), _torch_conv(x, w, s),
                                   rtol=1e-12, atol=1e-12)


def check_sizes(orc):
    """Window tensor vs im2col sizes (Sec. III-B).  The difference is
    N*C_i*K_h*H_o*(W_o*K_w - W_i) elements; when the filter tiles the width
    exactly (W_i = (W_o-1)*s + K_w) it is N*C_i*K_h*H_o*(W_o-1)*(K_w-s), which
    vanishes for s = K_w."""
    cases = [(int(a[1]), int(a[2]), int(a[3]), int(a[5]), int(a[6]), int(a[7]))
             for a in read_table("table1_layers.txt")]
    cases += [(3, 9, 9, 3, 3, 3), (2, 10, 10, 2, 2, 2), (4, 8, 11, 3, 2, 1), (5, 7, 7, 1, 1, 1)]
    for N in (1, 2):
        for Ci, H, W, Kh, Kw, s in cases:
            Ho, Wo = (H - Kh) // s + 1, (W - Kw) // s + 1
            assert orc.window_elems(N, Ci, H, W, Kh, s) == N * Ho * W * Kh * Ci
            assert orc.im2col_elems(N, Ci, H, W, Kh, Kw, s) == N * Ho * Wo * Kh * Kw * Ci
            diff = orc.im2col_elems(N, Ci, H, W, Kh, Kw, s) - orc.window_elems(N, Ci, H, W, Kh, s)
            assert diff == N * Ci * Kh * Ho * (Wo * Kw - W)
            if W == (Wo - 1) * s + Kw:
                assert diff == N * Ci * Kh * Ho * (Wo - 1) * (Kw - s)
                if s == Kw:
                    assert diff == 0
            # the window tensor is the smaller one whenever windows overlap
            if s < Kw and W == (Wo - 1) * s + Kw:
                assert diff > 0


def check_sizes_match_materialised(orc):
    for (N, Ci, H, W, Co, Kh, Kw, s) in TINY:
        x = np.zeros((N, H, W, Ci), np.float32)
        assert orc.im2win(x, Kh, s).size == orc.window_elems(N, Ci, H, W, Kh, s)


# Zero padding (an extension; the paper's layers have none), pinned against
# torch's padded conv2d, against the unpadded oracle on an explicitly padded
# input, and against closed forms.
PAD_CASES = [
    # N, Ci, H, W, Co, Kh, Kw, s, pad_h, pad_w
    (2, 3, 5, 6, 4, 3, 3, 1, 1, 1),     # "same" 3x3
    (1, 2, 7, 5, 3, 3, 2, 2, 2, 1),     # K_h != K_w, stride 2, pad_h != pad_w
    (2, 4, 4, 4, 2, 2, 3, 3, 0, 2),     # padding on one axis only
    (1, 1, 3, 2, 2, 2, 2, 1, 3, 3),     # pad larger than the filter: all-zero rims
    (3, 5, 6, 7, 6, 5, 5, 1, 2, 2),     # "same" 5x5
]


def _torch_conv_pad(x, w, s, ph, pw):
    xt = torch.from_numpy(np.ascontiguousarray(x, np.float64)).permute(0, 3, 1, 2)
    wt = torch.from_numpy(np.ascontiguousarray(w, np.float64)).permute(3, 2, 0, 1)
    y = torch.nn.functional.conv2d(xt, wt.contiguous(), stride=s, padding=(ph, pw))
    return y.permute(0, 2, 3, 1).contiguous().numpy()


def _zero_pad(x, ph, pw):
    return np.pad(x, ((0, 0), (ph, ph), (pw, pw), (0, 0)))


def check_pad_vs_torch_conv2d(orc):
    for t, (N, Ci, H, W, Co, Kh, Kw, s, ph, pw) in enumerate(PAD_CASES):
        r = _rng(60 + t)
        x = r.uniform(-1, 1, (N, H, W, Ci))
        w = r.uniform(-1, 1, (Kh, Kw, Ci, Co))
        y = orc.conv_pad(x, w, s, ph, pw)
        ref = _torch_conv_pad(x, w, s, ph, pw)
        assert y.shape == ref.shape, (y.shape, ref.shape)
        np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)


def check_pad_vs_explicit_zeros(orc):
    # integer inputs: the padded sum equals the unpadded sum over the padded
    # array exactly, and so does the |x||w| sum
    for t, (N, Ci, H, W, Co, Kh, Kw, s, ph, pw) in enumerate(PAD_CASES):
        r = _rng(70 + t)
        x = r.integers(-2, 3, (N, H, W, Ci)).astype(np.float64)
        w = r.integers(-2, 3, (Kh, Kw, Ci, Co)).astype(np.float64)
        y, a = orc.conv_pad(x, w, s, ph, pw, with_abs=True)
        ref = _slice_conv(_zero_pad(x, ph, pw), w, s)
        aref = _slice_conv(np.abs(_zero_pad(x, ph, pw)), np.abs(w), s)
        assert np.array_equal(y, ref) and np.array_equal(a, aref)


def check_pad_same_delta(orc):
    # centred delta filter with pad (K-1)/2 and stride 1: output = input
    for (K, Ci) in [(3, 2), (5, 3)]:
        x = _rng(80 + K).uniform(-1, 1, (2, 6, 5, Ci))
        w = np.zeros((K, K, Ci, Ci))
        for c in range(Ci):
            w[K // 2, K // 2, c, c] = 1.0
        y = orc.conv_pad(x, w, 1, K // 2, K // 2)
        assert np.array_equal(y, x)


def check_pad_zero_is_unpadded(orc):
    for t, (N, Ci, H, W, Co, Kh, Kw, s) in enumerate(TINY):
        r = _rng(90 + t)
        x = r.uniform(-1, 1, (N, H, W, Ci))
        w = r.uniform(-1, 1, (Kh, Kw, Ci, Co))
        assert np.array_equal(orc.conv_pad(x, w, s, 0, 0), orc.conv(x, w, s))
        x16 = x.astype(np.float16)
        assert orc.im2win_pad(x16, Kh, s, 0, 0).tobytes() == orc.im2win(x16, Kh, s).tobytes()


def check_im2win_pad_layout(orc):
    for t, (N, Ci, H, W, Co, Kh, Kw, s, ph, pw) in enumerate(PAD_CASES):
        r = _rng(100 + t)
        for dt in (np.float32, np.float16):
            x = r.uniform(-1, 1, (N, H, W, Ci)).astype(dt)
            win = orc.im2win_pad(x, Kh, s, ph, pw)
            assert win.dtype == dt
            assert win.tobytes() == _numpy_im2win(_zero_pad(x, ph, pw), Kh, s).tobytes()


# Filter dilation (an extension, combined with padding), pinned against
# torch's dilated conv2d, against the padded oracle with a zero-inserted filter
# (exact on integers), against d = 1 and 1x1 reductions, and a slicing-built
# window layout.
DIL_CASES = [
    # N, Ci, H, W, Co, Kh, Kw, s, pad_h, pad_w, d
    (2, 3, 9, 10, 4, 3, 3, 1, 2, 2, 2),     # "same" 3x3, d = 2
    (1, 2, 11, 9, 3, 3, 2, 2, 1, 3, 3),     # K_h != K_w, stride 2, d = 3, pad_h != pad_w
    (2, 4, 8, 8, 2, 2, 2, 1, 0, 0, 4),      # no padding, d = 4
    (1, 1, 7, 13, 2, 3, 3, 3, 0, 1, 2),     # stride 3 > d, padded width not a multiple of d
    (1, 3, 6, 6, 2, 1, 1, 1, 0, 0, 3),      # 1x1: dilation changes nothing
]


def _torch_conv_dil(x, w, s, ph, pw, d):
    xt = torch.from_numpy(np.ascontiguousarray(x, np.float64)).permute(0, 3, 1, 2)
    wt = torch.from_numpy(np.ascontiguousarray(w, np.float64)).permute(3, 2, 0, 1)
    y = torch.nn.functional.conv2d(xt, wt.contiguous(), stride=s, padding=(ph, pw), dilation=d)
    return y.permute(0, 2, 3, 1).contiguous().numpy()


def _insert_zeros(w, d):
    Kh, Kw, Ci, Co = w.shape
    big = np.zeros(((Kh - 1) * d + 1, (Kw - 1) * d + 1, Ci, Co), w.dtype)
    big[::d, ::d] = w
    return big


def check_dil_vs_torch_conv2d(orc):
    for t, (N, Ci, H, W, Co, Kh, Kw, s, ph, pw, d) in enumerate(DIL_CASES):
        r = _rng(110 + t)
        x = r.uniform(-1, 1, (N, H, W, Ci))
        w = r.uniform(-1, 1, (Kh, Kw, Ci, Co))
        y = orc.conv_dil(x, w, s, ph, pw, d)
        ref = _torch_conv_dil(x, w, s, ph, pw, d)
        assert y.shape == ref.shape, (y.shape, ref.shape)
        np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)


def check_dil_vs_inserted_zeros(orc):
    # integer inputs: the dilated filter is the filter with d-1 zero rows and
    # columns between taps; the padded oracle on it gives the same sums exactly
    for t, (N, Ci, H, W, Co, Kh, Kw, s, ph, pw, d) in enumerate(DIL_CASES):
        r = _rng(120 + t)
        x = r.integers(-2, 3, (N, H, W, Ci)).astype(np.float64)
        w = r.integers(-2, 3, (Kh, Kw, Ci, Co)).astype(np.float64)
        y, a = orc.conv_dil(x, w, s, ph, pw, d, with_abs=True)
        ref, aref = orc.conv_pad(x, _insert_zeros(w, d), s, ph, pw, with_abs=True)
        assert np.array_equal(y, ref) and np.array_equal(a, aref)


def check_dil_reductions(orc):
    # d = 1 is the padded convolution and window tensor; a 1x1 filter ignores d
    for t, (N, Ci, H, W, Co, Kh, Kw, s, ph, pw, d) in enumerate(DIL_CASES + [c[:10] + (1,) for c in DIL_CASES]):
        r = _rng(130 + t)
        x = r.uniform(-1, 1, (N, H, W, Ci))
        w = r.uniform(-1, 1, (Kh, Kw, Ci, Co))
        if d == 1:
            assert np.array_equal(orc.conv_dil(x, w, s, ph, pw, 1), orc.conv_pad(x, w, s, ph, pw))
            x16 = x.astype(np.float16)
            assert orc.im2win_dil(x16, Kh, s, ph, pw, 1).tobytes() == orc.im2win_pad(x16, Kh, s, ph, pw).tobytes()
        if Kh == 1 and Kw == 1:
            assert np.array_equal(orc.conv_dil(x, w, s, ph, pw, d), orc.conv_pad(x, w, s, ph, pw))


def check_im2win_dil_layout(orc):
    # every window is one contiguous span of its strip, holding the dilated
    # patch in (v, u, r) order; every padded column sits in exactly one strip
    # position of its residue group, the rest of the strip is zero
    for t, (N, Ci, H, W, Co, Kh, Kw, s, ph, pw, d) in enumerate(DIL_CASES):
        x = _rng(140 + t).uniform(-1, 1, (N, H, W, Ci)).astype(np.float32)
        xp = _zero_pad(x, ph, pw)
        Hp, Wp = xp.shape[1], xp.shape[2]
        win = orc.im2win_dil(x, Kh, s, ph, pw, d)
        Ho = orc.dil_extent(Hp, Kh, s, d)
        Wo = orc.dil_extent(Wp, Kw, s, d)
        Wq = -(-Wp // d)
        assert win.shape == (N, Ho, d * Wq * Kh, Ci)
        strips = win.reshape(N, Ho, d * Wq, Kh, Ci)
        seen = []
        for P in range(d * Wq):
            k = (P % Wq) * d + P // Wq
            if k < Wp:
                seen.append(k)
                for m in range(Ho):
                    rows = xp[:, m * s + np.arange(Kh) * d, k, :]
                    assert np.array_equal(strips[:, m, P], rows)
            else:
                assert not strips[:, :, P].any()
        assert sorted(seen) == list(range(Wp))
        flat = win.reshape(N, Ho, -1)
        T = Kh * Ci
        for m in range(Ho):
            for n in range(Wo):
                c0 = orc.dil_window_col(n, s, d, Wq)
                span = flat[:, m, c0 * T:(c0 + Kw) * T]
                patch = xp[:, m * s + np.arange(Kh)[None, :] * d, n * s + np.arange(Kw)[:, None] * d, :]
                assert np.array_equal(span, patch.reshape(N, -1)), (t, m, n)


def check_windowed_dil_equals_direct(orc):
    for t, (N, Ci, H, W, Co, Kh, Kw, s, ph, pw, d) in enumerate(DIL_CASES):
        r = _rng(150 + t)
        x = r.integers(-2, 3, (N, H, W, Ci)).astype(np.float64)
        w = r.integers(-2, 3, (Kh, Kw, Ci, Co)).astype(np.float64)
        win = orc.im2win_dil(x, Kh, s, ph, pw, d)
        y = orc.windowed_conv_dil(win, w, H + 2 * ph, W + 2 * pw, s, d)
        assert np.array_equal(y, orc.conv_dil(x, w, s, ph, pw, d))


ALL_CHECKS = [
    check_table1_extents, check_fig1_shapes, check_vs_torch_conv2d, check_vs_strided_slices,
    check_1x1_is_matmul, check_delta_filter, check_full_filter_is_dot, check_linearity,
    check_abs_sum, check_points, check_im2win_layout, check_im2win_identity,
    check_windows_contiguous, check_windowed_equals_direct, check_sizes,
    check_sizes_match_materialised, check_pad_vs_torch_conv2d, check_pad_vs_explicit_zeros,
    check_pad_same_delta, check_pad_zero_is_unpadded, check_im2win_pad_layout,
    check_dil_vs_torch_conv2d, check_dil_vs_inserted_zeros, check_dil_reductions, check_im2win_dil_layout,
    check_windowed_dil_equals_direct,
]

"""fp32 windowed convolution on the matrix cores (conv_im2win_fp32_mfma, an
alternate fp32 path) on the GPU against the fp64 oracle: the fp32 bar
(max |y - O| / sum|x||w| <= 1e-5), integer inputs exact, every tile variant,
every configured layer, non-finite inputs kept in their windows; layers with
C_i not a multiple of 4 take the vector-ALU kernel and must match it bit for
bit."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_20725_amd as pkg
from gpu_util import Run, TOL, check_sampled, oracle_inputs, rel_err, say
from test_gpu_conv import EDGE, _id
from paper_2608_20725_amd import workloads

pytestmark = pytest.mark.gpu

F32 = torch.float32


def _mfma_run(x, w, s):
    """Transform with the library, then the matrix-core fp32 conv into the
    NaN-poisoned, guarded output of a Run."""
    run = Run(x, w, s, F32, conv=False)
    pkg.conv_im2win_fp32_mfma(run.ws, run.wd, run.out, run.N, run.Ci, run.H, run.W, s)
    torch.cuda.synchronize()
    return run


def _check(run, x, w):
    xo, wo = oracle_inputs(x, w, F32)
    ref, absref = oracle.conv(xo, wo, run.s, with_abs=True)
    y = run.out_np()
    assert not np.isnan(y).any(), "output element left unwritten"
    r = rel_err(y, ref, absref)
    assert r <= TOL[F32], "max |err|/sum|x||w| = %.3g" % r
    return r


@pytest.mark.parametrize("shape", EDGE, ids=_id)
def test_fp32_mfma_edge_shapes(shape):
    N, Ci, H, W, Co, Kh, Kw, s = shape
    say("fp32 mfma", shape)
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=7 + sum(shape))
    run = _mfma_run(x, w, s)
    _check(run, x, w)
    run.check_out_guards()
    run.check_workspace_guard()
    if Ci % 4:   # the vector-ALU kernel runs: same bits as conv_im2win_fp32
        ref = Run(x, w, s, F32)
        assert torch.equal(run.out.view(torch.int32), ref.out.view(torch.int32))


@pytest.mark.parametrize("shape", EDGE[-19:], ids=_id)
def test_fp32_mfma_integer_inputs_exact(shape):
    N, Ci, H, W, Co, Kh, Kw, s = shape
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=11, dist="int2")
    run = _mfma_run(x, w, s)
    assert np.array_equal(run.out_np(), oracle.conv(x.double().numpy(), w.double().numpy(), s))


@pytest.mark.parametrize("layer", workloads.ALL, ids=lambda l: l.name)
def test_fp32_mfma_layers_small_batch(layer):
    x, w = workloads.draw_layer(layer, N=min(2, layer.N))
    run = _mfma_run(x, w, layer.stride)
    _check(run, x, w)
    run.check_out_guards()


@pytest.mark.parametrize("layer", workloads.ALL, ids=lambda l: l.name)
def test_fp32_mfma_layers_full_batch_sampled(layer):
    say("fp32 mfma full", layer.name)
    x, w = workloads.draw_layer(layer)
    run = _mfma_run(x, w, layer.stride)
    r, n = check_sampled(run, x, w, seed=layer.seed)
    say("  max rel err %.3g over %d outputs" % (r, n))
    run.check_out_guards()


@pytest.mark.parametrize("shape", [(2, 16, 13, 13, 72, 5, 5, 1), (2, 64, 24, 24, 300, 3, 3, 1),
                                   (3, 4, 13, 11, 33, 3, 3, 1)], ids=_id)
def test_fp32_mfma_tile_variants_agree(shape, monkeypatch):
    """Every tile accumulates the taps in the same order: same bits."""
    N, Ci, H, W, Co, Kh, Kw, s = shape
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=17)
    first = None
    for name in ("c128p128s2", "c64p256s2", "c32p256s2", "c64p128s2", "c32p128s2"):
        monkeypatch.setenv("IM2WIN_FP32_MFMA_TILE", name)
        run = _mfma_run(x, w, s)
        _check(run, x, w)
        run.check_out_guards()
        out = run.out.clone()
        if first is None:
            first = out
        else:
            assert torch.equal(out.view(torch.int32), first.view(torch.int32)), name


def test_fp32_mfma_deterministic():
    x, w = workloads.draw_layer(workloads.CFG2, N=4)
    a = _mfma_run(x, w, 1).out.clone()
    b = _mfma_run(x, w, 1).out.clone()
    assert torch.equal(a.view(torch.int32), b.view(torch.int32))


@pytest.mark.parametrize("shape", [(2, 16, 12, 14, 40, 3, 3, 1), (2, 8, 12, 14, 40, 5, 5, 1)], ids=_id)
def test_fp32_mfma_nonfinite_inputs_stay_in_their_windows(shape):
    N, Ci, H, W, Co, Kh, Kw, s = shape
    x, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=23)
    rng = np.random.default_rng(23)
    for v in (float("inf"), float("-inf"), float("nan")):
        x[rng.integers(N), rng.integers(H), rng.integers(W), rng.integers(Ci)] = v
    run = _mfma_run(x, w, s)
    with np.errstate(invalid="ignore", over="ignore"):
        ref, absref = oracle.conv(x.double().numpy(), w.double().numpy(), s, with_abs=True)
    y = run.out_np()
    fin = np.isfinite(ref)
    assert (~fin).any() and fin.any()
    assert np.array_equal(np.isfinite(y), fin)
    assert rel_err(y[fin], ref[fin], absref[fin]) <= TOL[F32]

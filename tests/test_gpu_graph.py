"""The path captured in a HIP graph (torch.cuda.graph over the C-ABI calls,
which launch on the current stream): every replay must reproduce the eager
result bit for bit, with eager work, input changes and synchronisations
between the replays (the library records no memset nodes: the transform
zeroes its pad with a kernel)."""
import pytest
import torch

import paper_2608_20725_amd as pkg
from gpu_util import say
from paper_2608_20725_amd import workloads

pytestmark = pytest.mark.gpu

CASES = [
    ((4, 64, 20, 20, 64, 3, 3, 1), torch.float32),
    ((4, 64, 20, 20, 64, 3, 3, 1), torch.float16),
    ((2, 3, 31, 29, 40, 5, 5, 2), torch.float32),   # unaligned windows: the element gather
    ((2, 3, 31, 29, 40, 5, 5, 2), torch.bfloat16),
    ((2, 256, 9, 9, 300, 3, 3, 1), torch.float16),   # several channel tiles, XCD-aware order
]


def _eager(x, w, s, dtype):
    N, H, W, Ci = x.shape
    Kh, Kw, _, Co = w.shape
    Ho, Wo = pkg.conv_output_dims(H, W, Kh, Kw, s)
    ws = torch.empty(pkg.conv_workspace_bytes(N, Ci, H, W, Co, Kh, Kw, s, dtype), dtype=torch.uint8, device="cuda")
    out = torch.empty((N, Ho, Wo, Co), dtype=dtype, device="cuda")
    pkg.conv_im2win_transform(x, ws, Co, Kh, Kw, s)
    pkg.conv_for_dtype(dtype)(ws, w, out, N, Ci, H, W, s)
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c[0])) + "-" + str(c[1])[6:])
def test_graph_replays_match_eager(case):
    (N, Ci, H, W, Co, Kh, Kw, s), dtype = case
    say("graph", case)
    xa, w = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=61)
    xb, _ = workloads.draw(N, Ci, H, W, Co, Kh, Kw, seed=62)
    xa, xb, w = xa.to(dtype).cuda(), xb.to(dtype).cuda(), w.to(dtype).cuda()
    ref_a, ref_b = _eager(xa, w, s, dtype), _eager(xb, w, s, dtype)
    bits = torch.int32 if dtype == torch.float32 else torch.int16
    assert not torch.equal(ref_a.view(bits), ref_b.view(bits))

    x = xa.clone()
    Ho, Wo = pkg.conv_output_dims(H, W, Kh, Kw, s)
    ws = torch.empty(pkg.conv_workspace_bytes(N, Ci, H, W, Co, Kh, Kw, s, dtype), dtype=torch.uint8, device="cuda")
    out = torch.empty((N, Ho, Wo, Co), dtype=dtype, device="cuda")
    conv = pkg.conv_for_dtype(dtype)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):   # one eager call on the capture stream first
        pkg.conv_im2win_transform(x, ws, Co, Kh, Kw, s)
        conv(ws, w, out, N, Ci, H, W, s)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, capture_error_mode="relaxed"):
        pkg.conv_im2win_transform(x, ws, Co, Kh, Kw, s)
        conv(ws, w, out, N, Ci, H, W, s)
    torch.cuda.synchronize()
    for rep, (src, ref) in enumerate([(xa, ref_a), (xa, ref_a), (xb, ref_b), (xa, ref_a)]):
        x.copy_(src)
        out.fill_(float("nan"))        # eager work between the replays
        ws[: ws.numel() // 2].zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(bits), ref.view(bits)), "replay %d" % rep

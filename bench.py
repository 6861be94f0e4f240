"""Benchmark of the im2win hot path on one MI355X.

One step = the whole path on one batch of synthetic input, in both
precisions the path has:
    fp32: im2win transform -> fp32 windowed conv (vector ALUs)
    fp16: im2win transform -> filter pack + fp16 windowed conv (MFMA, fp32 acc)
Default workload: N=128, C_i=64, H=W=56, C_o=64, 3x3, stride 1, uniform[-1,1]
values (seed 1), inputs resident in HBM before timing starts.

value = conv FLOPs of the step (2 * 2*N*H_o*W_o*C_o*K_h*K_w*C_i) / step time.
Per-kernel durations come from HIP events recorded on the stream the kernels
are launched on, around every call in the timed region.

Prints ONE JSON line.  `--layer NAME` picks another configured layer and
`--sweep` prints one line per configured layer instead (for reports);
`--ablation LAYERS` times the path with each of the paper's techniques
switched off (Sec. IV-D) on the named layers.  Each
line also carries a `bf16` block (the same layer with bf16 operands on the
same matrix-core kernels), an `fp32_mfma` block (the alternate fp32 path on
the matrix cores) and a `dilated` block (the layer with filter dilation 2 and
'same' padding, fp32 and fp16), all timed outside the step (extensions of the
path), a `cold` block (pack+conv with L2 and Infinity Cache flushed before
each call), a `clock` block (the shader clock sampled while the step
runs) and a `graph` block (the step captured in a HIP graph and replayed,
against call-by-call launches).
"""
from __future__ import annotations

import argparse
import json
import math
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# MI355X published peaks
PEAK_HBM_GBS = 8000.0
PEAK_FP32_VECTOR_TF = 157.3     # 256 CU x 256 flop/clk x 2.4 GHz (fp32 MFMA dense: the same)
PEAK_FP16_MFMA_TF = 2516.6      # dense (bf16 the same)

# HBM-side bytes per launch of the fp32 conv kernel, from rocprofv3 FETCH_SIZE and
# WRITE_SIZE counters (FETCH_SIZE scaled by 2.0 and WRITE_SIZE by 1.0, the
# factors a plain 1 GiB copy gives), keyed by layer.  They hold only for the
# kernel source they were taken on, identified by SHA-256 over FP32_SOURCES;
# after any change to those sources the figure is reported as null until
# measured again.  Source: profiles/cfg2_n128_c64_56_3x3.md.
FP32_SOURCES = ("conv_fp32_dma.hip",)
FP32_CONV_TRAFFIC = {
    "source_sha256": "17b1052a42de343bb699ff48f2307aa587a56aaa87f644e93853d0ced3ceaab2",
    "bytes": {"cfg2_n128_c64_56_3x3": 1016.6e6 + 95.6e6},
}


def fp32_sources_sha256():
    import hashlib
    h = hashlib.sha256()
    for name in FP32_SOURCES:
        with open(os.path.join(ROOT, "paper_2608_20725_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def fp32_conv_traffic(layer_name):
    if fp32_sources_sha256() != FP32_CONV_TRAFFIC["source_sha256"]:
        return None
    return FP32_CONV_TRAFFIC["bytes"].get(layer_name)


def layer_numbers(l, pkg):
    Ho, Wo = pkg.conv_output_dims(l.H, l.W, l.K_h, l.K_w, l.stride)
    P = l.N * Ho * Wo
    K = l.K_h * l.K_w * l.C_i
    flops = 2.0 * P * l.C_o * K
    d = {"Ho": Ho, "Wo": Wo, "P": P, "K": K, "flops": flops}
    for dt, elt in (("f32", 4), ("f16", 2)):
        win = l.N * Ho * l.W * l.K_h * l.C_i * elt
        d[dt] = {
            "window_bytes": win,
            "workspace_bytes": pkg.conv_workspace_bytes(l.N, l.C_i, l.H, l.W, l.C_o, l.K_h, l.K_w,
                                                        l.stride, dt),
            "im2col_bytes": pkg.conv_im2col_bytes(l.N, l.C_i, l.H, l.W, l.K_h, l.K_w, l.stride, dt),
            "input_bytes": l.N * l.H * l.W * l.C_i * elt,
            "filter_bytes": K * l.C_o * elt,
            "output_bytes": P * l.C_o * elt,
            # algorithmic traffic: read every window-tensor element, the filter
            # and write every output once
            "conv_bytes": win + K * l.C_o * elt + P * l.C_o * elt,
            # transform: read the input rows the windows use, write the window tensor
            "transform_bytes": l.N * ((Ho - 1) * l.stride + l.K_h) * l.W * l.C_i * elt + win,
        }
    return d


class Path:
    """Device buffers of one layer in one precision; `step()` runs transform + conv."""

    def __init__(self, l, x, w, dtype, pkg, torch):
        self.pkg, self.torch = pkg, torch
        self.l = l
        dev = torch.device("cuda")
        self.x = x.to(dtype).contiguous().to(dev)
        self.w = w.to(dtype).contiguous().to(dev)
        Ho, Wo = pkg.conv_output_dims(l.H, l.W, l.K_h, l.K_w, l.stride)
        need = pkg.conv_workspace_bytes(l.N, l.C_i, l.H, l.W, l.C_o, l.K_h, l.K_w, l.stride, dtype)
        self.ws = torch.empty(need, dtype=torch.uint8, device=dev)
        self.out = torch.empty((l.N, Ho, Wo, l.C_o), dtype=dtype, device=dev)
        self.conv = pkg.conv_for_dtype(dtype)

    def transform(self):
        l = self.l
        self.pkg.conv_im2win_transform(self.x, self.ws, l.C_o, l.K_h, l.K_w, l.stride)

    def run_conv(self):
        l = self.l
        self.conv(self.ws, self.w, self.out, l.N, l.C_i, l.H, l.W, l.stride)


def measure_minibatch(l, paths, pkg, torch, n_chunk=32, reps=10):
    """The mini-batch entry point on the same layer and buffers: chunks of
    `n_chunk` images alternating between two streams.
    Outside the timed step; reports its time per batch (HIP events on the main
    stream, which waits for every transform) and its workspace."""
    res = {"n_chunk": n_chunk, "two_streams": True}
    aux = torch.cuda.Stream()
    for name, p in paths.items():
        need = pkg.conv_chunked_workspace_bytes(l.N, l.C_i, l.H, l.W, l.C_o, l.K_h, l.K_w, l.stride,
                                                n_chunk, True, p.x.dtype)
        ws = torch.empty(need, dtype=torch.uint8, device="cuda")
        for _ in range(2):
            pkg.conv_im2win_chunked(p.x, p.w, p.out, ws, l.stride, n_chunk, aux_stream=aux)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            pkg.conv_im2win_chunked(p.x, p.w, p.out, ws, l.stride, n_chunk, aux_stream=aux)
        e1.record()
        torch.cuda.synchronize()
        res[name] = {"ms": round(e0.elapsed_time(e1) / reps, 5), "workspace_bytes": need,
                     "full_batch_workspace_bytes": p.ws.numel()}
        del ws
    return res


def measure_fp32_mfma(l, x, w, pkg, torch, reps=20):
    """The alternate fp32 path on the matrix cores (v_mfma_f32_32x32x2_f32) on
    the same layer, outside the timed step: median pack+conv time over `reps`
    runs, HIP events on the launch stream (layers with C_i not a multiple of
    4 run the vector-ALU kernel there)."""
    p = Path(l, x, w, torch.float32, pkg, torch)
    p.conv = pkg.conv_im2win_fp32_mfma
    p.transform()
    for _ in range(3):
        p.run_conv()
    torch.cuda.synchronize()
    ts = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        p.run_conv()
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1))
    ts.sort()
    Ho, Wo = pkg.conv_output_dims(l.H, l.W, l.K_h, l.K_w, l.stride)
    flops = 2.0 * l.N * Ho * Wo * l.C_o * l.K_h * l.K_w * l.C_i
    ms = ts[reps // 2]
    del p
    return {"pack_conv_ms": round(ms, 5), "TFLOP/s": round(flops / (ms * 1e-3) / 1e12, 3),
            "frac_fp32_mfma": round(flops / (ms * 1e-3) / 1e12 / PEAK_FP32_VECTOR_TF, 4),
            "on_matrix_cores": l.C_i % 4 == 0}


def measure_bf16(l, x, w, pkg, torch, reps=20):
    """The bf16 operand path (an extension beside the fp16 one: same kernels,
    bf16 MFMA) on the same layer, outside the timed step: median transform
    and pack+conv times over `reps` runs, HIP events on the launch stream."""
    p = Path(l, x, w, torch.bfloat16, pkg, torch)
    for _ in range(3):
        p.transform()
        p.run_conv()
    torch.cuda.synchronize()
    tr, cv = [], []
    for _ in range(reps):
        e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        e[0].record()
        p.transform()
        e[1].record()
        p.run_conv()
        e[2].record()
        torch.cuda.synchronize()
        tr.append(e[0].elapsed_time(e[1]))
        cv.append(e[1].elapsed_time(e[2]))
    tr.sort()
    cv.sort()
    Ho, Wo = pkg.conv_output_dims(l.H, l.W, l.K_h, l.K_w, l.stride)
    flops = 2.0 * l.N * Ho * Wo * l.C_o * l.K_h * l.K_w * l.C_i
    ms_t, ms_c = tr[reps // 2], cv[reps // 2]
    del p
    return {"transform_ms": round(ms_t, 5), "pack_conv_ms": round(ms_c, 5),
            "TFLOP/s": round(flops / (ms_c * 1e-3) / 1e12, 3),
            "frac_bf16_mfma": round(flops / (ms_c * 1e-3) / 1e12 / PEAK_FP16_MFMA_TF, 4)}


# The paper's ablation (Sec. IV-D, Table II) on its three tensor-core
# techniques, mapped to their gfx950 counterparts; each entry switches one off
# through the library's tuning variables (read at every launch).
ABLATION = {
    "f16": [
        ("as built", {}),
        ("no column reuse: row-per-pixel kernel", {"IM2WIN_FP16_KERNEL": "pipe"}),
        ("row kernel 128x128, 2-slot ring", {"IM2WIN_FP16_KERNEL": "pipe", "IM2WIN_FP16_TILE": "c128p128s2"}),
        ("row kernel 128x128, 1 slot (no double buffering)",
         {"IM2WIN_FP16_KERNEL": "pipe", "IM2WIN_FP16_TILE": "c128p128s1"}),
        ("register-staged loads (no direct-to-LDS copy)", {"IM2WIN_FP16_KERNEL": "regs"}),
        ("launch-order tiles (no XCD-aware tile order)", {"IM2WIN_TILE_ORDER": "linear"}),
    ],
    "f32": [
        ("as built", {}),
        ("register-staged loads (no direct-to-LDS copy)", {"IM2WIN_FP32_KERNEL": "regs"}),
        ("launch-order tiles (no XCD-aware tile order)", {"IM2WIN_TILE_ORDER": "linear"}),
    ],
    "transform": [
        ("as built (XCD-aware block order)", {}),
        ("linear block order", {"IM2WIN_TRANSFORM_ORDER": "linear"}),
    ],
}
ABLATION_VARS = ("IM2WIN_FP16_KERNEL", "IM2WIN_FP16_TILE", "IM2WIN_FP32_KERNEL", "IM2WIN_TRANSFORM_ORDER",
                 "IM2WIN_TILE_ORDER")


def run_ablation(l, pkg, torch, workloads, reps=9, rounds=5):
    """Time of each call of the path with one technique switched off, on
    layer `l`.  The variants are interleaved so that clock ramps and drift
    fall on all of them alike: after an untimed pass over every variant,
    `rounds` passes each time `reps` back-to-back calls (warm caches) of
    every variant, in reverse order on every other pass; the figure is the
    median over the passes of each pass's median."""
    x, w = workloads.draw_layer(l)
    paths = {"f32": Path(l, x, w, torch.float32, pkg, torch),
             "f16": Path(l, x, w, torch.float16, pkg, torch)}
    nums = layer_numbers(l, pkg)
    for p in paths.values():
        p.transform()   # the window tensor the conv variants read

    cases = []   # (part, label, environment, call, bytes moved or None)
    for part, rows in ABLATION.items():
        for label, env in rows:
            if part == "transform":
                for dt in ("f32", "f16"):
                    cases.append((part, "%s %s" % (dt, label), env, paths[dt].transform,
                                  nums[dt]["transform_bytes"]))
            else:
                cases.append((part, label, env, paths[part].run_conv, None))

    def set_env(env):
        for k in ABLATION_VARS:
            os.environ.pop(k, None)
        os.environ.update(env)

    def timed(fn, n):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(n):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        return statistics.median(ts)

    times = {c[1] + "\0" + c[0]: [] for c in cases}
    saved = {k: os.environ.get(k) for k in ABLATION_VARS}
    try:
        for _, _, env, fn, _ in cases:
            set_env(env)
            timed(fn, reps)
        for r in range(rounds):
            for part, label, env, fn, _ in (cases if r % 2 == 0 else cases[::-1]):
                set_env(env)
                times[label + "\0" + part].append(timed(fn, reps))
    finally:
        for k, v in saved.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v
    res = {"layer": l.name, "rounds": rounds, "reps": reps, "f16": {}, "f32": {}, "transform": {}}
    for part, label, _, _, nbytes in cases:
        ms = statistics.median(times[label + "\0" + part])
        if nbytes is not None:
            res[part][label] = {"ms": round(ms, 5), "GB/s": round(nbytes / ms / 1e6, 1)}
        else:
            res[part][label] = {"ms": round(ms, 5), "TFLOP/s": round(nums["flops"] / (ms * 1e-3) / 1e12, 2)}
    del paths
    return res


def measure_dilated(l, x, w, pkg, torch, d=2, reps=20):
    """The atrous version of the layer (filter dilation d, zero padding
    d*(K-1)/2 so the output keeps the input extent when the stride is 1), in
    fp32 and fp16, outside the timed step: median transform and pack+conv
    times over `reps` runs, HIP events on the launch stream, and the window
    tensor against an im2col matrix of the same layer."""
    ph, pw = d * (l.K_h - 1) // 2, d * (l.K_w - 1) // 2
    Hp, Wp = l.H + 2 * ph, l.W + 2 * pw
    Ho, Wo = pkg.conv_output_dims_dilated(Hp, Wp, l.K_h, l.K_w, l.stride, d)
    flops = 2.0 * l.N * Ho * Wo * l.C_o * l.K_h * l.K_w * l.C_i
    res = {"dilation": d, "pad": [ph, pw], "output": [Ho, Wo]}
    for name, dt in (("f32", torch.float32), ("f16", torch.float16)):
        xd = x.to(dt).contiguous().cuda()
        wd = w.to(dt).contiguous().cuda()
        need = pkg.conv_workspace_bytes_dilated(l.N, l.C_i, Hp, Wp, l.C_o, l.K_h, l.K_w, l.stride, d, dt)
        ws = torch.empty(need, dtype=torch.uint8, device="cuda")
        out = torch.empty((l.N, Ho, Wo, l.C_o), dtype=dt, device="cuda")

        def tr():
            pkg.conv_im2win_transform_dilated(xd, ws, l.C_o, l.K_h, l.K_w, l.stride, ph, pw, d)

        def cv():
            pkg.conv_im2win_dilated(ws, wd, out, l.N, l.C_i, Hp, Wp, l.stride, d)
        for _ in range(3):
            tr()
            cv()
        torch.cuda.synchronize()
        t_tr, t_cv = [], []
        for _ in range(reps):
            e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
            e[0].record()
            tr()
            e[1].record()
            cv()
            e[2].record()
            torch.cuda.synchronize()
            t_tr.append(e[0].elapsed_time(e[1]))
            t_cv.append(e[1].elapsed_time(e[2]))
        t_tr.sort()
        t_cv.sort()
        elt = 4 if dt == torch.float32 else 2
        im2col = l.N * Ho * Wo * l.K_h * l.K_w * l.C_i * elt
        win = l.N * Ho * d * ((Wp + d - 1) // d) * l.K_h * l.C_i * elt
        res[name] = {"transform_ms": round(t_tr[reps // 2], 5), "pack_conv_ms": round(t_cv[reps // 2], 5),
                     "TFLOP/s": round(flops / (t_cv[reps // 2] * 1e-3) / 1e12, 3),
                     "window_bytes": win, "im2col_bytes": im2col, "window_over_im2col": round(win / im2col, 4)}
        del xd, wd, ws, out
    return res


def cpu_baseline(l, x, w, budget_s=10.0):
    """The fp64 oracle on the host cores over whole images of the same layer,
    a few images at a time, cycling through the batch until `budget_s` has
    elapsed (a bounded sample; the rate is per image, so the count of images
    done fixes the work)."""
    import oracle
    oracle.build()
    xs = x.double().numpy()
    wd = w.double().numpy()
    Ho = (l.H - l.K_h) // l.stride + 1
    Wo = (l.W - l.K_w) // l.stride + 1
    per_img = 2.0 * Ho * Wo * l.C_o * l.K_h * l.K_w * l.C_i
    done, t0 = 0, time.perf_counter()
    chunk = 4
    while time.perf_counter() - t0 < budget_s:
        i0 = done % l.N
        n = min(chunk, l.N - i0)
        oracle.conv(xs[i0:i0 + n], wd, l.stride)
        done += n
    dt = time.perf_counter() - t0
    cores = oracle.threads()
    # one image on one thread
    oracle.set_threads(1)
    try:
        t1 = time.perf_counter()
        oracle.conv(xs[:1], wd, l.stride)
        dt1 = time.perf_counter() - t1
    finally:
        oracle.set_threads(cores)
    return {"value": per_img * done / dt / 1e12, "unit": "TFLOP/s", "cores": cores,
            "kind": "oracle",
            "sample": "%d images (%.1f passes over the batch of %d) of the same layer, fp64 direct "
                      "convolution, %.1f s" % (done, done / l.N, l.N, dt),
            "single_thread": {"value": per_img / dt1 / 1e12, "unit": "TFLOP/s", "seconds": round(dt1, 3),
                              "sample": "1 image of the same layer on 1 thread"}}


def measure_graph(l, paths, nums, torch, reps=50):
    """The step (both transforms and both pack+conv calls) captured once in a
    HIP graph and replayed: time per step over `reps` back-to-back replays
    (HIP events around the whole loop), against the same step launched call
    by call.  The library launches on the current stream, so capture records
    its kernels; it records no memset nodes."""
    def step():
        for name in ("f32", "f16"):
            paths[name].transform()
            paths[name].run_conv()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, capture_error_mode="relaxed"):
        step()
    torch.cuda.synchronize()
    res = {"reps": reps}
    for name, fn in (("graph", g.replay), ("eager", step)):
        for _ in range(10):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        res[name] = {"ms_per_step": round(ms, 5), "TFLOP/s": round(2 * nums["flops"] / (ms * 1e-3) / 1e12, 3)}
    del g
    return res


def measure_cold(l, paths, nums, torch, reps=10):
    """Pack+conv time with cold caches: before each timed call a 1 GiB
    buffer is overwritten (untimed), which evicts the window tensor and the
    filter from L2 and the 256 MB Infinity Cache; median of `reps` calls,
    HIP events on the launch stream."""
    flush = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
    res = {"flush_bytes": flush.numel() * 4, "reps": reps}
    for name, p in paths.items():
        p.transform()
        ts = []
        for r in range(reps):
            flush.fill_(float(r))
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            p.run_conv()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        ms = statistics.median(ts)
        res[name] = {"ms": round(ms, 5), "min_ms": round(min(ts), 5),
                     "TFLOP/s": round(nums["flops"] / (ms * 1e-3) / 1e12, 3)}
    del flush
    return res


def measure(l, steps, warmup, pkg, torch, workloads):
    x, w = workloads.draw_layer(l)
    paths = {"f32": Path(l, x, w, torch.float32, pkg, torch),
             "f16": Path(l, x, w, torch.float16, pkg, torch)}
    nums = layer_numbers(l, pkg)

    def step(ev=None):
        for k, name in enumerate(("f32", "f16")):
            p = paths[name]
            if ev is not None:
                ev[3 * k].record()
            p.transform()
            if ev is not None:
                ev[3 * k + 1].record()
            p.run_conv()
            if ev is not None:
                ev[3 * k + 2].record()

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        step(evs[i])
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0

    def avg(a, b):
        v = sorted(evs[i][a].elapsed_time(evs[i][b]) for i in range(steps))
        return sum(v) / len(v), v[0], v[len(v) // 2]

    k = {}
    for j, name in enumerate(("f32", "f16")):
        k[name + "_transform_ms"] = avg(3 * j, 3 * j + 1)
        k[name + "_conv_ms"] = avg(3 * j + 1, 3 * j + 2)
    k["clock"] = sample_clock(step, torch)
    return nums, k, elapsed, x, w, paths


def sample_clock(step, torch, seconds=1.5, settle=0.5, period=0.01):
    """Shader clock while the step runs: after the timed region, untimed
    steps of the same workload for `seconds`, with a background thread
    reading each XCD's current gfx clock (amdsmi GPU metrics, which the
    driver refreshes every few tens of ms) every `period` seconds; samples
    from the first `settle` seconds are dropped.  Returns an "error" entry
    when amdsmi is unusable."""
    import threading
    try:
        import amdsmi
        amdsmi.amdsmi_init()
    except Exception as e:   # no amdsmi on this host: report, do not fail
        return {"error": "amdsmi unavailable: %s" % e}
    samples = []
    try:
        handles = amdsmi.amdsmi_get_processor_handles()
        h = handles[torch.cuda.current_device()] if len(handles) == torch.cuda.device_count() else handles[0]
        stop = threading.Event()
        t0 = time.perf_counter()

        def run():
            while not stop.is_set():
                m = amdsmi.amdsmi_get_gpu_metrics_info(h)
                c = [v for v in m.get("current_gfxclks", []) if isinstance(v, int) and v < 0xFFFF]
                if c and time.perf_counter() - t0 >= settle:
                    samples.append(c)
                stop.wait(period)
        th = threading.Thread(target=run, daemon=True)
        th.start()
        n = 0
        while time.perf_counter() - t0 < seconds:
            for _ in range(20):
                step()
            n += 20
            torch.cuda.synchronize()
        stop.set()
        th.join()
    except Exception as e:
        return {"error": "amdsmi: %s" % e}
    finally:
        try:
            amdsmi.amdsmi_shut_down()
        except Exception:
            pass
    if not samples:
        return {"error": "no clock samples"}
    mean = sorted(sum(c) / len(c) for c in samples)
    per = [statistics.median(c[j] for c in samples) for j in range(min(len(c) for c in samples))]
    return {"MHz_median": round(statistics.median(mean)), "MHz_min": round(mean[0]), "MHz_max": round(mean[-1]),
            "per_xcd_median_MHz": [round(v) for v in per], "samples": len(samples),
            "source": "amdsmi current_gfxclks (mean over XCDs) during %d untimed steps (%.1f s) after the "
                      "timed region, first %.1f s dropped" % (n, seconds, settle)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    # the clock takes a few tens of steps to settle after the inputs are drawn
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--layer", default=None, help="configured layer name (default: cfg2)")
    ap.add_argument("--sweep", action="store_true", help="one line per configured layer")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--ablation", default=None, metavar="LAYERS",
                    help="comma-separated layer names: time the path with each of the paper's "
                         "techniques switched off (one JSON line per layer) and exit")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="BYTES",
                    help="only run a plain device-to-device copy of BYTES bytes (HBM counter "
                         "calibration) and exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the im2win path runs on a single MI355X here "
              "(batch sharding across GPUs is described, not built); use --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    import torch
    if args.calibrate_copy:
        src = torch.ones(args.calibrate_copy // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(max(args.steps, 1)):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": src.numel() * 4, "copies": max(args.steps, 1)}), flush=True)
        return
    import paper_2608_20725_amd as pkg
    from paper_2608_20725_amd import workloads

    if not os.path.exists(pkg.library_path()):
        from paper_2608_20725_amd import build
        build.build()
    pkg.load_library()

    if args.ablation:
        for name in args.ablation.split(","):
            print(json.dumps(run_ablation(workloads.BY_NAME[name], pkg, torch, workloads)), flush=True)
            torch.cuda.empty_cache()
        return

    layers = list(workloads.ALL) if args.sweep else [
        workloads.BY_NAME[args.layer] if args.layer else workloads.CFG2]
    for l in layers:
        torch.cuda.reset_peak_memory_stats()
        nums, k, elapsed, x, w, paths = measure(l, args.steps, args.warmup, pkg, torch, workloads)
        peak_alloc = torch.cuda.max_memory_allocated()
        ms = elapsed / args.steps * 1e3
        flops = nums["flops"]
        value = 2 * flops / (ms * 1e-3) / 1e12
        c32 = k["f32_conv_ms"][0]
        c16 = k["f16_conv_ms"][0]
        t32 = k["f32_transform_ms"][0]
        t16 = k["f16_transform_ms"][0]
        tf32 = flops / (c32 * 1e-3) / 1e12
        tf16 = flops / (c16 * 1e-3) / 1e12
        f32, f16 = nums["f32"], nums["f16"]
        rec = {
            "metric": "conv TFLOPS (fp32 VALU, fp16 MFMA) + peak workspace bytes vs im2col",
            "value": round(value, 3),
            "unit": "TFLOP/s",
            "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
            "ms_per_step": round(ms, 4),
            "higher_is_better": True,
            "scaling": "weak",
            "vs_baseline": None,
            "dtype": "f32+f16(f32acc)",
            "data": "synthetic",
            "config": {"workload": "%s: N=%d C_i=%d H=W=%d C_o=%d %dx%d stride %d, %s values, "
                                   "fp32 and fp16 paths" % (l.name, l.N, l.C_i, l.H, l.C_o, l.K_h,
                                                            l.K_w, l.stride, l.dist),
                       "global_batch": l.N, "parallelism": "single GPU"},
            "roofline": {
                "kernel": "conv_fp32_dma (fp32 windowed conv, VALU)",
                "bound": "alu",
                "achieved": round(tf32, 3),
                "peak": PEAK_FP32_VECTOR_TF,
                "unit": "TFLOP/s",
                "frac": round(tf32 / PEAK_FP32_VECTOR_TF, 4),
                "traffic": fp32_conv_traffic(l.name),
            },
            "kernels": {
                "f32_transform": {"ms": round(t32, 5), "GB/s": round(f32["transform_bytes"] / t32 / 1e6, 1),
                                  "frac_hbm": round(f32["transform_bytes"] / t32 / 1e6 / PEAK_HBM_GBS, 4)},
                "f32_conv": {"ms": round(c32, 5), "TFLOP/s": round(tf32, 3),
                             "frac_fp32_vector": round(tf32 / PEAK_FP32_VECTOR_TF, 4),
                             "GB/s": round(f32["conv_bytes"] / c32 / 1e6, 1)},
                "f16_transform": {"ms": round(t16, 5), "GB/s": round(f16["transform_bytes"] / t16 / 1e6, 1),
                                  "frac_hbm": round(f16["transform_bytes"] / t16 / 1e6 / PEAK_HBM_GBS, 4)},
                "f16_pack_conv": {"ms": round(c16, 5), "TFLOP/s": round(tf16, 3),
                                  "frac_fp16_mfma": round(tf16 / PEAK_FP16_MFMA_TF, 4),
                                  "GB/s": round(f16["conv_bytes"] / c16 / 1e6, 1),
                                  "frac_hbm": round(f16["conv_bytes"] / c16 / 1e6 / PEAK_HBM_GBS, 4)},
                "median_ms": {n: round(v[2], 5) for n, v in k.items() if n != "clock"},
                "min_ms": {n: round(v[1], 5) for n, v in k.items() if n != "clock"},
            },
            "end_to_end_TFLOP/s": {"f32": round(flops / ((t32 + c32) * 1e-3) / 1e12, 3),
                                   "f16": round(flops / ((t16 + c16) * 1e-3) / 1e12, 3)},
            "workspace": {
                "f32_window_bytes": f32["window_bytes"], "f32_im2col_bytes": f32["im2col_bytes"],
                "f32_window_over_im2col": round(f32["window_bytes"] / f32["im2col_bytes"], 4),
                "f16_window_bytes": f16["window_bytes"], "f16_im2col_bytes": f16["im2col_bytes"],
                "f16_workspace_bytes": f16["workspace_bytes"],
                "f16_workspace_over_im2col": round(f16["workspace_bytes"] / f16["im2col_bytes"], 4),
                "allocator_peak_bytes": peak_alloc,
            },
        }
        rec["clock"] = k["clock"]
        if "MHz_median" in rec["clock"]:
            # the fp32 conv against the vector peak at the clock it ran at
            rec["clock"]["f32_conv_frac_at_clock"] = round(
                tf32 / (PEAK_FP32_VECTOR_TF * rec["clock"]["MHz_median"] / 2400.0), 4)
        rec["bf16"] = measure_bf16(l, x, w, pkg, torch)
        rec["fp32_mfma"] = measure_fp32_mfma(l, x, w, pkg, torch)
        rec["dilated"] = measure_dilated(l, x, w, pkg, torch)
        rec["cold"] = measure_cold(l, paths, nums, torch)
        rec["graph"] = measure_graph(l, paths, nums, torch)
        if not args.sweep:
            mb = measure_minibatch(l, paths, pkg, torch)
            for name in ("f32", "f16"):
                full_ms = k[name + "_transform_ms"][0] + k[name + "_conv_ms"][0]
                mb[name]["TFLOP/s"] = round(flops / (mb[name]["ms"] * 1e-3) / 1e12, 3)
                mb[name]["full_batch_ms"] = round(full_ms, 5)
            rec["minibatch"] = mb
        if not args.no_cpu_baseline and not args.sweep:
            rec["cpu_baseline"] = cpu_baseline(l, x, w)
        print(json.dumps(rec), flush=True)
        del paths
        torch.cuda.empty_cache()


if __name__ == "__main__":
    main()

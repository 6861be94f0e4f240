"""Benchmark of the im2win hot path on one MI355X.

Workload (default): the 12-layer sweep at batch 128 -- the shapes of the
paper's benchmark table (Table I layers cv1, cv3-cv12) plus a 1x1 layer with
1024 channels -- in both precisions the path has, seeded synthetic values,
inputs resident in HBM before timing starts.  One step runs, for every layer
in turn:
    fp32: im2win transform -> fp32 windowed conv (vector ALUs)
    fp16: im2win transform -> filter pack + fp16 windowed conv (MFMA, fp32 acc)
W untimed warm-up steps, then K timed steps between two device
synchronisations.  Every call in the timed region is bracketed by HIP events
on the stream it is launched on (created without the system-scope fence, so
recording them leaves the caches and the kernels' timing alone).

value = conv-only throughput of the step in both precisions:
    sum over layers and precisions of 2*N*H_o*W_o*C_o*K_h*K_w*C_i
    / sum of the conv calls' average durations (pack + conv kernels).
The fp32 and fp16 figures are reported separately (`conv_only`), each with a
roofline block (`roofline`: fp32 vector ALUs, the kernel that dominates the
step; `roofline_f16`: fp16 matrix cores, with the attainable rate of each
layer's own bound), per-layer figures in `layers`, the kernel each call ran,
the transforms, the workspace against an im2col buffer (formula and measured
allocator peaks), the shader clock during the timed steps and the CPU oracle
on a bounded sample of the same workload.

After the timed region (outside it): the deep layer (N=128, 512 channels at
14x14) timed the same way, the sweep with bf16 operands and with fp32 on the
matrix cores, and the mini-batch entry point; `--no-extras` skips them.

`--layer NAME` times one configured layer instead of the sweep; `--ablation
LAYERS` times the path with each of the paper's techniques switched off
(Sec. IV-D) and exits; `--calibrate-copy BYTES` runs a plain device copy (for
HBM counter calibration) and exits.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import statistics
import sys
import threading
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# MI355X published peaks
PEAK_HBM_GBS = 8000.0
PEAK_FP32_VECTOR_TF = 157.3     # 256 CU x 256 flop/clk x 2.4 GHz (fp32 MFMA dense: the same)
PEAK_FP16_MFMA_TF = 2516.6      # dense (bf16 the same)

METRIC = "conv TFLOPS (fp32 VALU, fp16 MFMA) + peak workspace bytes vs im2col"

# HBM-side bytes per step moved by the conv kernels of the sweep, from
# rocprofv3 FETCH_SIZE and WRITE_SIZE (KiB per dispatch) over the timed
# dispatches of `bench.py --steps 20 --warmup 5`, each scaled by what the same
# counter reads for a plain device copy of known size.  They hold only for the
# kernel sources they were taken on (SHA-256 over KERNEL_SOURCES); after any
# change to those sources the figure is reported as null until measured again.
KERNEL_SOURCES = ("common.hpp", "epilogue16.hpp", "mfma16.hpp", "conv_fp32_dma.hip", "conv_fp32.hip",
                  "conv_fp32_stem.hip", "conv_fp16.hip", "conv_fp16_col.hip", "conv_fp16_seg.hip",
                  "conv_fp16_stem.hip")
CONV_TRAFFIC = {
    "source_sha256": "e20dbaf2266bb33c36af0556f974d8f62bd7eae1206a88acc5975f318ac1bd83",
    "workload": "sweep",
    "f32": 16539423713,    # bytes per step, fetched + written
    "f16": 6495587517,
}


def kernel_sources_sha256():
    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2608_20725_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def conv_traffic(workload, dt):
    if CONV_TRAFFIC["workload"] != workload or CONV_TRAFFIC["source_sha256"] != kernel_sources_sha256():
        return None
    return CONV_TRAFFIC[dt]


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def layer_numbers(l, pkg):
    Ho, Wo = pkg.conv_output_dims(l.H, l.W, l.K_h, l.K_w, l.stride)
    P = l.N * Ho * Wo
    K = l.K_h * l.K_w * l.C_i
    flops = 2.0 * P * l.C_o * K
    d = {"Ho": Ho, "Wo": Wo, "P": P, "K": K, "flops": flops}
    for dt, elt in (("f32", 4), ("f16", 2)):
        win = l.N * Ho * l.W * l.K_h * l.C_i * elt
        conv_bytes = win + K * l.C_o * elt + P * l.C_o * elt
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
            "conv_bytes": conv_bytes,
            # transform: read the input rows the windows use, write the window tensor
            "transform_bytes": l.N * ((Ho - 1) * l.stride + l.K_h) * l.W * l.C_i * elt + win,
            "kernel": pkg.conv_im2win_kernel_name(l.N, l.C_i, l.H, l.W, l.C_o, l.K_h, l.K_w, l.stride, dt),
        }
    # fp16 roofline of the layer: the matrix cores, or HBM where the
    # algorithmic bytes at 8 TB/s take longer than the FLOPs at peak
    t_mfma = flops / (PEAK_FP16_MFMA_TF * 1e12)
    t_hbm = d["f16"]["conv_bytes"] / (PEAK_HBM_GBS * 1e9)
    d["f16"]["bound"] = "mfma" if t_mfma >= t_hbm else "hbm"
    d["f16"]["attainable_s"] = max(t_mfma, t_hbm)
    return d


class Path:
    """Device buffers of one layer in one precision: `transform()` and
    `run_conv()` call the C ABI on the current stream."""

    def __init__(self, l, x, w, dtype, pkg, torch, conv=None):
        self.pkg, self.torch = pkg, torch
        self.l = l
        dev = torch.device("cuda")
        self.x = x.to(dtype).contiguous().to(dev)
        self.w = w.to(dtype).contiguous().to(dev)
        Ho, Wo = pkg.conv_output_dims(l.H, l.W, l.K_h, l.K_w, l.stride)
        need = pkg.conv_workspace_bytes(l.N, l.C_i, l.H, l.W, l.C_o, l.K_h, l.K_w, l.stride, dtype)
        self.ws = torch.empty(need, dtype=torch.uint8, device=dev)
        self.out = torch.empty((l.N, Ho, Wo, l.C_o), dtype=dtype, device=dev)
        self.conv = conv or pkg.conv_for_dtype(dtype)

    def transform(self):
        l = self.l
        self.pkg.conv_im2win_transform(self.x, self.ws, l.C_o, l.K_h, l.K_w, l.stride)

    def run_conv(self):
        l = self.l
        self.conv(self.ws, self.w, self.out, l.N, l.C_i, l.H, l.W, l.stride)


class ClockSampler:
    """Shader clock of each XCD read through amdsmi (GPU metrics, which the
    driver refreshes every few tens of ms) every `period` seconds from a
    background thread while the timed steps run."""

    def __init__(self, torch, period=0.005):
        self.samples, self.error, self.period = [], None, period
        self.stop = threading.Event()
        try:
            import amdsmi
            amdsmi.amdsmi_init()
            handles = amdsmi.amdsmi_get_processor_handles()
            self.h = handles[torch.cuda.current_device()] if len(handles) == torch.cuda.device_count() \
                else handles[0]
            self.amdsmi = amdsmi
        except Exception as e:   # no amdsmi on this host: report, do not fail
            self.error = "amdsmi unavailable: %s" % e
            self.amdsmi = None

    def _run(self):
        while not self.stop.is_set():
            try:
                m = self.amdsmi.amdsmi_get_gpu_metrics_info(self.h)
                c = [v for v in m.get("current_gfxclks", []) if isinstance(v, int) and v < 0xFFFF]
                if c:
                    self.samples.append(c)
            except Exception as e:
                self.error = "amdsmi: %s" % e
                return
            self.stop.wait(self.period)

    def __enter__(self):
        if self.amdsmi is not None:
            self.th = threading.Thread(target=self._run, daemon=True)
            self.th.start()
        return self

    def __exit__(self, *exc):
        if self.amdsmi is not None:
            self.stop.set()
            self.th.join()
            try:
                self.amdsmi.amdsmi_shut_down()
            except Exception:
                pass

    def report(self):
        if not self.samples:
            return {"error": self.error or "no clock samples"}
        mean = sorted(sum(c) / len(c) for c in self.samples)
        per = [statistics.median(c[j] for c in self.samples) for j in range(min(len(c) for c in self.samples))]
        return {"MHz_median": round(statistics.median(mean)), "MHz_min": round(mean[0]),
                "MHz_max": round(mean[-1]), "per_xcd_median_MHz": [round(v) for v in per],
                "samples": len(self.samples),
                "source": "amdsmi current_gfxclks (mean over XCDs), sampled during the timed steps"}


def measure_workspace(l, pkg, torch):
    """Device bytes the caching allocator holds at its peak for one
    transform + conv of the layer (input, filter, output, workspace), against
    the same with the workspace replaced by a full-batch im2col buffer
    (N*H_o*W_o rows of K_h*K_w*C_i elements), per precision.  Buffers are
    allocated, measured and freed one set at a time."""
    res = {}
    for name, dt in (("f32", torch.float32), ("f16", torch.float16)):
        Ho, Wo = pkg.conv_output_dims(l.H, l.W, l.K_h, l.K_w, l.stride)
        need = pkg.conv_workspace_bytes(l.N, l.C_i, l.H, l.W, l.C_o, l.K_h, l.K_w, l.stride, dt)
        im2col = pkg.conv_im2col_bytes(l.N, l.C_i, l.H, l.W, l.K_h, l.K_w, l.stride, dt)
        peaks = {}
        for kind, nbytes in (("im2win", need), ("im2col", im2col)):
            torch.cuda.synchronize()
            base = torch.cuda.memory_allocated()
            torch.cuda.reset_peak_memory_stats()
            bufs = [torch.empty((l.N, l.H, l.W, l.C_i), dtype=dt, device="cuda"),
                    torch.empty((l.K_h, l.K_w, l.C_i, l.C_o), dtype=dt, device="cuda"),
                    torch.empty((l.N, Ho, Wo, l.C_o), dtype=dt, device="cuda"),
                    torch.empty(nbytes, dtype=torch.uint8, device="cuda")]
            peaks[kind] = torch.cuda.max_memory_allocated() - base
            del bufs
        res[name] = {"window_bytes": l.N * Ho * l.W * l.K_h * l.C_i * (4 if name == "f32" else 2),
                     "workspace_bytes": need, "im2col_bytes": im2col,
                     "im2col_bytes_per_image": im2col // l.N,
                     "window_over_im2col": round(l.N * Ho * l.W * l.K_h * l.C_i / (im2col / (4 if name == "f32"
                                                                                           else 2)), 4),
                     "workspace_over_im2col": round(need / im2col, 4),
                     "peak_bytes_im2win": peaks["im2win"], "peak_bytes_im2col": peaks["im2col"],
                     "peak_ratio": round(peaks["im2win"] / peaks["im2col"], 4)}
    torch.cuda.empty_cache()
    return res


class HipEvents:
    """HIP timing events recorded on torch's current stream (the stream the
    library launches on), created with hipEventDisableSystemFence: recording
    one then writes a timestamp without the system-scope fence (a cache
    write-back and invalidate) that a default event adds, which would idle
    the GPU for several microseconds at each event and start the next kernel
    with cold caches.  The device is synchronised before times are read."""

    _lib = None

    def __init__(self, torch):
        import ctypes
        if HipEvents._lib is None:
            # the HIP runtime torch has loaded (same soname, so the same copy)
            lib = ctypes.CDLL("libamdhip64.so.7")
            lib.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
            lib.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
            lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
            lib.hipEventDestroy.argtypes = [ctypes.c_void_p]
            HipEvents._lib = lib
        self.ctypes, self.torch = ctypes, torch
        self.events = []

    def new(self):
        ev = self.ctypes.c_void_p()
        rc = self._lib.hipEventCreateWithFlags(self.ctypes.byref(ev), 0x20000000)  # hipEventDisableSystemFence
        if rc != 0:
            raise RuntimeError("hipEventCreateWithFlags failed: %d" % rc)
        self.events.append(ev)
        return _Event(self, ev)

    def destroy(self):
        for ev in self.events:
            self._lib.hipEventDestroy(ev)
        self.events = []


class _Event:
    def __init__(self, owner, ev):
        self.owner, self.ev = owner, ev

    def record(self):
        st = self.owner.torch.cuda.current_stream().cuda_stream
        rc = self.owner._lib.hipEventRecord(self.ev, self.owner.ctypes.c_void_p(st))
        if rc != 0:
            raise RuntimeError("hipEventRecord failed: %d" % rc)

    def elapsed_time(self, other):
        ms = self.owner.ctypes.c_float()
        rc = self.owner._lib.hipEventElapsedTime(self.owner.ctypes.byref(ms), self.ev, other.ev)
        if rc != 0:
            raise RuntimeError("hipEventElapsedTime failed: %d" % rc)
        return ms.value


def timed_steps(step, nevents, steps, warmup, torch, clock=None):
    """`warmup` untimed steps, then `steps` timed ones between two device
    synchronisations; `step(ev)` records its events into the list `ev` of
    `nevents` HIP events.  Returns (wall seconds of the timed steps, events
    per step)."""
    for _ in range(warmup):
        step(None)
    hip = HipEvents(torch)
    evs = [[hip.new() for _ in range(nevents)] for _ in range(steps)]
    torch.cuda.synchronize()
    ctx = clock if clock is not None else _Null()
    with ctx:
        t0 = time.perf_counter()
        for i in range(steps):
            step(evs[i])
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t0
    return elapsed, evs


class _Null:
    def __enter__(self):
        return self

    def __exit__(self, *exc):
        return False


def mean_ms(evs, a, b):
    return sum(e[a].elapsed_time(e[b]) for e in evs) / len(evs)


def run_workload(layers, steps, warmup, pkg, torch, workloads):
    """The timed region: every layer, fp32 then fp16, transform then conv."""
    paths, nums, samples = [], [], []
    for l in layers:
        log("setup", l.name)
        x, w = workloads.draw_layer(l)
        paths.append({"f32": Path(l, x, w, torch.float32, pkg, torch),
                      "f16": Path(l, x, w, torch.float16, pkg, torch)})
        nums.append(layer_numbers(l, pkg))
        # image 0 and the filter, fp64, for the CPU oracle's sample
        samples.append((x[0:1].double().numpy(), w.double().numpy()))
        del x, w
    n = len(layers)

    def step(ev):
        for j, p in enumerate(paths):
            for k, name in enumerate(("f32", "f16")):
                b = 6 * j + 3 * k
                if ev is not None:
                    ev[b].record()
                p[name].transform()
                if ev is not None:
                    ev[b + 1].record()
                p[name].run_conv()
                if ev is not None:
                    ev[b + 2].record()

    clock = ClockSampler(torch)
    log("timed region: %d warm-up + %d steps" % (warmup, steps))
    elapsed, evs = timed_steps(step, 6 * n, steps, warmup, torch, clock)
    per = []
    for j in range(n):
        r = {}
        for k, name in enumerate(("f32", "f16")):
            b = 6 * j + 3 * k
            r[name] = {"transform_ms": mean_ms(evs, b, b + 1), "conv_ms": mean_ms(evs, b + 1, b + 2),
                       "conv_ms_min": min(e[b + 1].elapsed_time(e[b + 2]) for e in evs)}
        per.append(r)
    return paths, nums, samples, per, elapsed, clock.report()


def layer_record(l, nm, t):
    """Per-layer figures from the numbers `nm` and the times `t`."""
    rec = {"layer": l.name, "shape": {"N": l.N, "C_i": l.C_i, "H": l.H, "W": l.W, "C_o": l.C_o, "K": l.K_h,
                                      "stride": l.stride}, "GFLOP": round(nm["flops"] / 1e9, 3)}
    for name in ("f32", "f16"):
        d, tt = nm[name], t[name]
        tf = nm["flops"] / (tt["conv_ms"] * 1e-3) / 1e12
        r = {"kernel": d["kernel"], "conv_ms": round(tt["conv_ms"], 5), "TFLOP/s": round(tf, 2),
             "transform_ms": round(tt["transform_ms"], 5),
             "transform_GB/s": round(d["transform_bytes"] / tt["transform_ms"] / 1e6, 1),
             "conv_GB/s": round(d["conv_bytes"] / tt["conv_ms"] / 1e6, 1)}
        if name == "f32":
            r["frac_peak"] = round(tf / PEAK_FP32_VECTOR_TF, 4)
        else:
            att = nm["flops"] / d["attainable_s"] / 1e12
            r.update({"frac_peak": round(tf / PEAK_FP16_MFMA_TF, 4), "bound": d["bound"],
                      "attainable_TFLOP/s": round(att, 1), "frac_attainable": round(tf / att, 4)})
        rec[name] = r
    return rec


def aggregate(nums, per):
    """Sweep totals per precision: FLOPs over summed conv time."""
    res = {}
    for name, peak in (("f32", PEAK_FP32_VECTOR_TF), ("f16", PEAK_FP16_MFMA_TF)):
        flops = sum(nm["flops"] for nm in nums)
        ms = sum(t[name]["conv_ms"] for t in per)
        tf = flops / (ms * 1e-3) / 1e12
        per_layer = [nm["flops"] / (t[name]["conv_ms"] * 1e-3) / 1e12 for nm, t in zip(nums, per)]
        r = {"TFLOP/s": round(tf, 3), "frac_peak": round(tf / peak, 4), "conv_ms_per_step": round(ms, 5),
             "GFLOP_per_step": round(flops / 1e9, 6),
             "geomean_TFLOP/s": round(math.exp(sum(math.log(v) for v in per_layer) / len(per_layer)), 3),
             "algorithmic_bytes_per_step": sum(nm[name]["conv_bytes"] for nm in nums)}
        if name == "f16":
            att_s = sum(nm["f16"]["attainable_s"] for nm in nums)
            r["attainable_TFLOP/s"] = round(flops / att_s / 1e12, 1)
            r["frac_attainable"] = round(att_s / (ms * 1e-3), 4)
        res[name] = r
    return res


def cpu_baseline(layers, samples, budget_s=12.0):
    """The fp64 oracle on the host cores over whole images of the workload:
    one image of every layer in turn (`samples[j]` = image 0 and the filter
    of layer j, as the GPU got them), round after round until `budget_s` has
    passed -- a bounded sample of the same workload; the rate is the FLOPs
    done over the time taken.  One image of the first layer is also timed on
    one thread."""
    import oracle
    oracle.build()
    per_img = []
    for l in layers:
        Ho = (l.H - l.K_h) // l.stride + 1
        Wo = (l.W - l.K_w) // l.stride + 1
        per_img.append(2.0 * Ho * Wo * l.C_o * l.K_h * l.K_w * l.C_i)
    done, rounds = 0.0, 0
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < budget_s:
        for j, l in enumerate(layers):
            oracle.conv(samples[j][0], samples[j][1], l.stride)
            done += per_img[j]
        rounds += 1
    dt = time.perf_counter() - t0
    cores = oracle.threads()
    oracle.set_threads(1)
    try:
        t1 = time.perf_counter()
        oracle.conv(samples[0][0], samples[0][1], layers[0].stride)
        dt1 = time.perf_counter() - t1
    finally:
        oracle.set_threads(cores)
    return {"value": done / dt / 1e12, "unit": "TFLOP/s", "cores": cores, "kind": "oracle",
            "sample": "%d rounds of one whole image of each of the %d layers (image 0, the GPU's inputs), "
                      "fp64 direct convolution, %.1f s" % (rounds, len(layers), dt),
            "single_thread": {"value": per_img[0] / dt1 / 1e12, "unit": "TFLOP/s", "seconds": round(dt1, 3),
                              "sample": "1 image of %s on 1 thread" % layers[0].name}}


def conv_only_sweep(paths, nums, steps, warmup, torch, pkg, dtype, conv=None):
    """Conv calls only, over every layer, in another precision or on other
    kernels (outside the timed region): the window tensors are written once,
    then `warmup` untimed and `steps` timed passes over the layers' convs."""
    ps = [Path(p["f32"].l, p["f32"].x, p["f32"].w, dtype, pkg, torch, conv=conv) for p in paths]
    for p in ps:
        p.transform()

    def step(ev):
        for j, p in enumerate(ps):
            if ev is not None:
                ev[2 * j].record()
            p.run_conv()
            if ev is not None:
                ev[2 * j + 1].record()
    _, evs = timed_steps(step, 2 * len(ps), steps, warmup, torch)
    flops = sum(nm["flops"] for nm in nums)
    ms = [mean_ms(evs, 2 * j, 2 * j + 1) for j in range(len(ps))]
    res = {"TFLOP/s": round(flops / (sum(ms) * 1e-3) / 1e12, 3),
           "layers": {p.l.name: round(nm["flops"] / (t * 1e-3) / 1e12, 2) for p, nm, t in zip(ps, nums, ms)}}
    del ps
    torch.cuda.empty_cache()
    return res


def measure_minibatch(l, pkg, torch, workloads, steps, warmup, n_chunk=32):
    """The mini-batch entry point (chunks of `n_chunk` images alternating
    between two streams) on layer `l`, against the full-batch transform +
    conv pair: time per batch (HIP events on the main stream, which waits for
    the aux stream at the end of each call) and workspace bytes."""
    x, w = workloads.draw_layer(l)
    aux = torch.cuda.Stream()
    res = {"layer": l.name, "n_chunk": n_chunk, "two_streams": True}
    flops = layer_numbers(l, pkg)["flops"]
    for name, dt in (("f32", torch.float32), ("f16", torch.float16)):
        full = Path(l, x, w, dt, pkg, torch)
        need = pkg.conv_chunked_workspace_bytes(l.N, l.C_i, l.H, l.W, l.C_o, l.K_h, l.K_w, l.stride,
                                                n_chunk, True, dt)
        ws = torch.empty(need, dtype=torch.uint8, device="cuda")

        def chunked(ev):
            if ev is not None:
                ev[0].record()
            pkg.conv_im2win_chunked(full.x, full.w, full.out, ws, l.stride, n_chunk, aux_stream=aux)
            if ev is not None:
                ev[1].record()

        def whole(ev):
            if ev is not None:
                ev[0].record()
            full.transform()
            full.run_conv()
            if ev is not None:
                ev[1].record()
        _, e1 = timed_steps(chunked, 2, steps, warmup, torch)
        _, e2 = timed_steps(whole, 2, steps, warmup, torch)
        ms, ms_full = mean_ms(e1, 0, 1), mean_ms(e2, 0, 1)
        res[name] = {"ms": round(ms, 5), "TFLOP/s": round(flops / (ms * 1e-3) / 1e12, 3),
                     "kernel": pkg.conv_im2win_kernel_name(n_chunk, l.C_i, l.H, l.W, l.C_o, l.K_h, l.K_w,
                                                           l.stride, dt),
                     "workspace_bytes": need, "full_batch_ms": round(ms_full, 5),
                     "full_batch_workspace_bytes": full.ws.numel()}
        del full, ws
    torch.cuda.empty_cache()
    return res


def roofline_blocks(agg, workload):
    f32, f16 = agg["f32"], agg["f16"]
    r32 = {"kernel": "fp32 windowed conv on the vector ALUs (conv_fp32_dma, conv_fp32_stem), all layers of the step",
           "bound": "alu", "achieved": f32["TFLOP/s"], "peak": PEAK_FP32_VECTOR_TF, "unit": "TFLOP/s",
           "frac": round(f32["TFLOP/s"] / PEAK_FP32_VECTOR_TF, 4), "traffic": conv_traffic(workload, "f32"),
           "per": "step (one conv call per layer; achieved = algorithmic FLOPs / summed average durations)",
           "algorithmic_bytes": f32["algorithmic_bytes_per_step"]}
    r16 = {"kernel": "fp16 windowed conv on the matrix cores (fp32 accumulation), all layers of the step",
           "bound": "mfma", "achieved": f16["TFLOP/s"], "peak": PEAK_FP16_MFMA_TF, "unit": "TFLOP/s",
           "frac": round(f16["TFLOP/s"] / PEAK_FP16_MFMA_TF, 4), "traffic": conv_traffic(workload, "f16"),
           "attainable": f16["attainable_TFLOP/s"], "frac_attainable": f16["frac_attainable"],
           "per": "step (one conv call per layer; attainable = FLOPs / sum over layers of max(FLOPs / peak, "
                  "algorithmic bytes / 8 TB/s))",
           "algorithmic_bytes": f16["algorithmic_bytes_per_step"]}
    return r32, r16

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




def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--layer", default=None, help="one configured layer as the workload (default: the sweep)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the blocks measured after the timed region")
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

    if args.layer:
        layers = [workloads.BY_NAME[args.layer]]
        workload = args.layer
        wdesc = "%s: N=%d C_i=%d H=W=%d C_o=%d %dx%d stride %d, %s values, fp32 and fp16 paths" % (
            layers[0].name, layers[0].N, layers[0].C_i, layers[0].H, layers[0].C_o, layers[0].K_h,
            layers[0].K_w, layers[0].stride, layers[0].dist)
    else:
        layers = list(workloads.SWEEP)
        workload = "sweep"
        wdesc = ("sweep of 12 conv layers at N=128 (Table I layers cv1, cv3-cv12 and a 1x1 C=1024 layer; "
                 "S1-S12), fp32 and fp16 paths, seeded uniform[-1,1] values")

    wsp = [measure_workspace(l, pkg, torch) for l in layers]
    paths, nums, samples, per, elapsed, clock = run_workload(layers, args.steps, args.warmup, pkg, torch,
                                                             workloads)
    ms_step = elapsed / args.steps * 1e3
    agg = aggregate(nums, per)
    flops_step = 2 * sum(nm["flops"] for nm in nums)
    conv_ms = agg["f32"]["conv_ms_per_step"] + agg["f16"]["conv_ms_per_step"]
    value = flops_step / (conv_ms * 1e-3) / 1e12
    r32, r16 = roofline_blocks(agg, workload)
    tr = {}
    for name in ("f32", "f16"):
        b = sum(nm[name]["transform_bytes"] for nm in nums)
        t = sum(p[name]["transform_ms"] for p in per)
        tr[name] = {"ms_per_step": round(t, 5), "GB/s": round(b / t / 1e6, 1),
                    "frac_hbm": round(b / t / 1e6 / PEAK_HBM_GBS, 4)}
    rec = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32+f16(f32acc)",
        "data": "synthetic",
        "config": {"workload": wdesc, "layers": [l.name for l in layers], "global_batch": layers[0].N,
                   "parallelism": "single GPU"},
        "value_is": "conv-only TFLOP/s of the step, both precisions: conv FLOPs / summed average conv-call "
                    "durations (HIP events); per precision in conv_only",
        "conv_only": agg,
        "roofline": r32,
        "roofline_f16": r16,
        "end_to_end_TFLOP/s": round(flops_step / (ms_step * 1e-3) / 1e12, 3),
        "transform": tr,
        "layers": [layer_record(l, nm, t) for l, nm, t in zip(layers, nums, per)],
        "workspace": {l.name: w for l, w in zip(layers, wsp)},
        "clock": clock,
    }
    if "MHz_median" in clock:
        # the conv rates against the peaks scaled to the clock they ran at
        rec["clock"]["f32_frac_at_clock"] = round(
            agg["f32"]["TFLOP/s"] / (PEAK_FP32_VECTOR_TF * clock["MHz_median"] / 2400.0), 4)
        rec["clock"]["f16_frac_at_clock"] = round(
            agg["f16"]["TFLOP/s"] / (PEAK_FP16_MFMA_TF * clock["MHz_median"] / 2400.0), 4)
    if not args.no_extras:
        ext = {}
        log("extras: bf16 and fp32 on the matrix cores over the workload")
        ext["bf16"] = conv_only_sweep(paths, nums, args.steps, args.warmup, torch, pkg, torch.bfloat16)
        ext["fp32_matrix_cores"] = conv_only_sweep(paths, nums, args.steps, args.warmup, torch, pkg, torch.float32,
                                                   conv=pkg.conv_im2win_fp32_mfma)
        del paths
        torch.cuda.empty_cache()
        if workload == "sweep":
            log("extras: the deep layer")
            cfg4 = workloads.CFG4
            p4, n4, _, t4, _, _ = run_workload([cfg4], args.steps, args.warmup, pkg, torch, workloads)
            ext["cfg4"] = layer_record(cfg4, n4[0], t4[0])
            del p4
            torch.cuda.empty_cache()
            log("extras: mini-batch")
            ext["minibatch"] = measure_minibatch(workloads.CFG2, pkg, torch, workloads, args.steps, args.warmup)
        rec["extras"] = ext
    else:
        del paths
    if not args.no_cpu_baseline:
        log("cpu baseline")
        rec["cpu_baseline"] = cpu_baseline(layers, samples)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()

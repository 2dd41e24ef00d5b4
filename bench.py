#!/usr/bin/env python3
"""Benchmark of the SINGA hot path on one MI355X.

One step = BPTrainOneBatch (Alg. 1) plus the Updater on the AlexNet-shaped
training workload: batch 256 of 3x227x227 images, bf16 compute with fp32
accumulation and fp32 master weights, conv 96x11x11/4 - maxpool - conv
256x5x5 - maxpool - conv 384x3x3 - conv 384x3x3 - conv 256x3x3 - maxpool -
FC 9216-4096-4096-1000 (ReLU after every conv and the first two FC),
softmax cross-entropy over random labels, and one fused SGD-momentum update
(lr 0.01, momentum 0.9, weight decay 5e-4) of all 62,378,344 parameters.
Inputs are seeded synthetic tensors resident in HBM before timing starts.

The step runs the filter gradients of the convolution layers on a second
stream, beside the backward-data passes (--single-stream: one stream).

Timing follows the paper's protocol by default (Sec. 6.2.2: run 100
iterations, average iterations 30-80): 30 warm-up steps, then 50 timed steps
between two device synchronizations, twice: replays of a HIP graph holding
one whole step, and the same steps launched eagerly (--eager: eager only).
`value` is the faster of the two (`launch` says which; both are reported).
Then the same number of steps runs eagerly on one stream with the library's
kernel trace on, which brackets every launch with HIP events: each kernel
runs alone on the GPU, and the per-kernel figures (and the roofline of the
dominant kernel) come from those.  A rocprofv3 summary whose average
durations match these comes from a --single-stream run.  Last, the step runs
for one more second while a side thread reads the graphics clock (amdsmi),
and the MFMA roofline is also priced at the clock measured (`sclk`).

Prints one JSON line.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK = {"bf16_tflops": 2516.6, "f32_tflops": 157.3, "hbm_gbs": 8000.0}
METRIC = "conv fwd+bwd TFLOP/s (% MFMA peak) and training images/sec, 1×MI355X"
# the GEMM kernels of the conv / FC passes (each tagged with its layer pass's
# algorithmic flops) and the helper kernels those passes launch
CONV_KERNELS = ("conv_fwd_kernel", "conv_fwd_large_kernel", "conv_wgrad_kernel", "conv_wgrad_large_kernel",
                "bwd_data_direct_kernel")
CONV_HELPERS = ("transpose_kernel", "transpose_vec_kernel", "splitk_reduce_kernel", "splitk_epilogue_kernel",
                "splitk_epilogue_vec_kernel", "pad_channels_kernel", "unpad_channels_f32_kernel",
                "space_to_depth_kernel", "filter_to_s2d_kernel", "s2d_to_filter_f32_kernel",
                "depth_to_space_kernel")


def is_conv_kernel(name):
    """A conv / FC GEMM kernel (the name up to its template arguments)."""
    return name.split("<")[0] in CONV_KERNELS


def is_conv_helper(name):
    return name.split("<")[0] in CONV_HELPERS


def step_conv_flops(w, batch, need_input_grad=False):
    """Algorithmic flops of the conv / FC passes of one step of workload w:
    2 x the multiply-adds of the direct definition (padded taps included) for
    the forward pass, the filter gradient and the input gradient of every
    layer, except the first layer's input gradient, which training does not
    need (counted only with need_input_grad)."""
    from paper_1603_07846_amd import workloads as wl
    total = 0.0
    c, h, ww = w.in_shape
    first = True
    for l in w.layers:
        if isinstance(l, (wl.Conv, wl.FC)):
            k, p, q = l.out_shape
            r, s = (l.kernel, l.kernel) if isinstance(l, wl.Conv) else (h, ww)
            one = 2.0 * batch * p * q * k * c * r * s
            total += one * (3 if (not first or need_input_grad) else 2)
            first = False
        if isinstance(l, (wl.Conv, wl.Pool, wl.FC)):
            c, h, ww = l.out_shape
    return total


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=30)
    ap.add_argument("--workload", type=int, default=5, help="workload index (5 = AlexNet-shaped training step)")
    ap.add_argument("--eager", action="store_true", help="time eager launches only (no graph replays)")
    ap.add_argument("--single-stream", action="store_true",
                    help="run every pass on one stream (no concurrent filter gradients), as the per-kernel pass does")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-images", type=int, default=40, help="images in the oracle's timed sample (about 10 s on 16 cores)")
    ap.add_argument("--steps-only", action="store_true",
                    help="only the timed and traced steps (no clock reading, Updater / LRN lines, other workloads or "
                         "CPU baseline): the short run the counter passes profile")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the other workloads' lines (single layer, CIFAR-shaped net, fp32 / bf16 conv stacks)")
    return ap.parse_args()


def measured_traffic(kernel):
    """HBM bytes per launch of `kernel` from the committed counter summary
    (profiles/traffic.json: FETCH_SIZE + WRITE_SIZE per dispatch, calibrated
    against a copy of known size), or None when there is none for this kernel
    or its source file has changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    from paper_1603_07846_amd.profiling import sha256_of
    with open(path) as f:
        t = json.load(f)
    src = os.path.join(ROOT, t.get("source", ""))
    if t.get("kernel") != kernel or not os.path.exists(src) or sha256_of(src) != t.get("source_sha256"):
        return None
    return round(t["bytes_per_launch"])


class GfxClock:
    """Reads the GPU's current graphics clock (SCLK, MHz) through the amdsmi
    library while the step runs, so the MFMA peak (quoted at 2400 MHz) can also
    be priced at the clock the kernels actually ran at.  The reading lags the
    load by a hundred milliseconds or more (it can still show the idle clock
    through a whole 50-step timed region that ran at full speed), so the clock
    is taken over a separate run of the same steps after the timed regions,
    from its second half.  Any failure (no amdsmi, no permission, several GPUs
    with no match) leaves the figures null; it never stops the benchmark."""

    NOMINAL_MHZ = 2400.0

    def __init__(self, period_s=0.005):
        self.period = period_s
        self.h = None
        self.err = None
        self.vals = []
        self.window = None
        try:
            import amdsmi
            self.smi = amdsmi
            amdsmi.amdsmi_init(amdsmi.AmdSmiInitFlags.INIT_AMD_GPUS)
            hs = amdsmi.amdsmi_get_processor_handles()
            if len(hs) == 1:
                self.h = hs[0]
            else:
                import torch
                p = torch.cuda.get_device_properties(0)
                want = (getattr(p, "pci_domain_id", 0), getattr(p, "pci_bus_id", -1), getattr(p, "pci_device_id", -1))
                for h in hs:
                    dom, rest = amdsmi.amdsmi_get_gpu_device_bdf(h).split(":", 1)
                    bus, devfn = rest.split(":")
                    if (int(dom, 16), int(bus, 16), int(devfn.split(".")[0], 16)) == want:
                        self.h = h
                if self.h is None:
                    self.err = "%d GPUs visible to amdsmi and none matches device 0" % len(hs)
            if self.h is not None:
                self.read()
        except Exception as e:  # noqa: BLE001 - any failure only disables the figure
            self.h, self.err = None, "%s: %s" % (type(e).__name__, (str(e).strip().splitlines() or [""])[-1].strip())

    def read(self):
        return float(self.smi.amdsmi_get_clock_info(self.h, self.smi.AmdSmiClkType.GFX)["clk"])

    def steady(self, step, seconds=1.0, settle=0.5):
        """Runs step() back to back for `seconds` while a side thread reads the
        clock every period; keeps the readings taken after `settle` seconds."""
        import threading
        import torch
        if self.h is None:
            return
        got, stop = [], threading.Event()
        t0 = time.perf_counter()

        def loop():
            while not stop.is_set():
                try:
                    got.append((time.perf_counter() - t0, self.read()))
                except Exception:  # noqa: BLE001
                    return
                stop.wait(self.period)

        t = threading.Thread(target=loop, daemon=True)
        t.start()
        try:
            n = 0
            while time.perf_counter() - t0 < seconds:
                step()
                n += 1
                if n % 8 == 0:  # bound the queue so the window is time on the GPU
                    torch.cuda.synchronize()
            torch.cuda.synchronize()
        finally:
            stop.set()
            t.join()
        self.vals = [v for ts, v in got if ts >= settle]
        self.window = (seconds, settle, n)

    def mhz(self):
        return sum(self.vals) / len(self.vals) if self.vals else None

    def summary(self):
        if not self.vals:
            return {"error": self.err or "no readings"}
        return {"mhz_mean": round(self.mhz(), 1), "mhz_min": min(self.vals), "mhz_max": max(self.vals),
                "samples": len(self.vals), "nominal_mhz": self.NOMINAL_MHZ,
                "source": "amdsmi current GFX clock every %g ms over the last %g s of a %g s run of %d eager "
                          "steps after the timed regions" % (self.period * 1e3, self.window[0] - self.window[1],
                                                             self.window[0], self.window[2])}


CONFIG_NAMES = {1: "single_conv_layer_fwd_bwd_sgd_f32_b16", 2: "cifar_convnet_train_step_f32_b100",
                3: "alexnet_conv_stack_fwd_bwd_f32_b128", 4: "alexnet_conv_stack_fwd_bwd_bf16_b256"}


# images of each smaller workload in its oracle sample
CONFIG_CPU_IMAGES = {1: 16, 2: 100, 3: 4, 4: 4}


def measure_config(index, steps, warmup):
    """One of the other workloads, timed on its own: `steps` eager steps
    between two device synchronizations after `warmup` untimed ones (the
    single-layer workload also computes its input gradient, as its three
    passes define it), the same number replayed from a HIP graph of one step
    (the faster of the two is the workload's step time), then the same steps
    launched eagerly with the kernel trace on.  The
    step's algorithmic conv / FC flops over the step time and over the
    summed conv-kernel time, against the peak of the workload's dtype."""
    import torch
    from paper_1603_07846_amd import net as gnet
    from paper_1603_07846_amd import singa
    from paper_1603_07846_amd import workloads as wl

    w = wl.WORKLOADS[index]
    dev = torch.device("cuda:0")
    inp = wl.make_inputs(w)
    net = gnet.Net(w, device=dev)
    net.load_params(inp.params)
    x = net.to_device_input(inp.x)
    labels = torch.from_numpy(inp.labels).to(dev) if inp.labels is not None else None
    dy = net.to_device_input(inp.dy) if inp.dy is not None else None
    need_dx = index == 1

    def step():
        net.train_one_batch(x, labels=labels, dy_top=dy, need_input_grad=need_dx)

    def timed(fn):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            fn()
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) * 1e3 / steps

    for _ in range(warmup):
        step()
    eager_ms = timed(step)
    # the same steps replayed from a HIP graph of one step (these small steps
    # are launch-bound: replay issues all their kernels at once)
    graph = net.capture(x, labels=labels, dy_top=dy, need_input_grad=need_dx)
    for _ in range(3):
        graph.replay()
    graph_ms = timed(graph.replay)
    del graph
    ms = min(eager_ms, graph_ms)
    side = net.wgrad_stream
    net.wgrad_stream = None
    singa.trace_enable(True)
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    singa.trace_enable(False)
    net.wgrad_stream = side
    recs = singa.trace_records()
    traced_flops = sum(r[2] for r in recs if is_conv_kernel(r[0])) / steps
    conv_ms = sum(r[1] for r in recs if is_conv_kernel(r[0]) or is_conv_helper(r[0])) / steps
    flops = step_conv_flops(w, net.batch, need_dx)
    peak = PEAK["bf16_tflops"] if w.dtype == "bf16" else PEAK["f32_tflops"]
    tf_step = flops / (ms / 1e3) / 1e12
    tf_conv = flops / (conv_ms / 1e3) / 1e12
    out = {"workload": CONFIG_NAMES[index], "description": w.name, "dtype": w.dtype, "batch": net.batch,
           "ms_per_step": round(ms, 4), "images_per_s": round(net.batch / (ms / 1e3), 1),
           "launch": "eager" if eager_ms <= graph_ms else "hip_graph", "eager_ms_per_step": round(eager_ms, 4),
           "graph_ms_per_step": round(graph_ms, 4),
           "conv_gflop_per_step": round(flops / 1e9, 4), "traced_conv_gflop_per_step": round(traced_flops / 1e9, 4),
           "tflops_over_step": round(tf_step, 3), "frac_peak_over_step": round(tf_step / peak, 4),
           "conv_kernel_ms_per_step": round(conv_ms, 4), "tflops_over_conv_kernels": round(tf_conv, 3),
           "frac_peak_over_conv_kernels": round(tf_conv / peak, 4), "peak_tflops": peak,
           "steps": steps, "warmup": warmup}
    del net, x, labels, dy
    torch.cuda.empty_cache()
    return out


def measure_updaters(net, w):
    """Both Updater protocols over the whole flat parameter buffer, each
    alone, timed with HIP events (on a copy of the net's buffers, so the
    step's state is left as it was)."""
    import torch
    from paper_1603_07846_amd import singa
    updaters = {}
    wf, gf, vf = net.w_flat.clone(), net.g_flat.clone(), torch.zeros_like(net.v_flat)
    wbf = net.wb_flat.clone() if net.wb_flat is not None else None
    nbytes = net.n_params_padded * (22 if wbf is not None else 20)
    for name, fn in (("sgd_momentum", lambda: singa.sgd_momentum_update(wf, gf, vf, wbf, w.lr, w.momentum,
                                                                        w.weight_decay)),
                     ("adagrad", lambda: singa.adagrad_update(wf, gf, vf, wbf, w.lr, 1e-6, w.weight_decay))):
        for _ in range(3):
            fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(20):
            fn()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / 20
        updaters[name] = {"ms": round(ms, 4), "GB_per_s": round(nbytes / (ms / 1e3) / 1e9, 1),
                          "frac_hbm_peak": round(nbytes / (ms / 1e3) / 1e9 / PEAK["hbm_gbs"], 4),
                          "params": net.n_params_padded}
    del wf, gf, vf, wbf
    return updaters


def measure_lrn(net, dev, is_bf16):
    """Local response normalization (not part of this step: the paper's GPU
    AlexNet leaves it out) at the two AlexNet positions, batch 256, alone."""
    import torch
    from paper_1603_07846_amd import singa
    lrn = {}
    gen = torch.Generator(device=dev)
    gen.manual_seed(1603078465)
    dt_t = torch.bfloat16 if is_bf16 else torch.float32
    es = 2 if is_bf16 else 4
    for name, (C, H) in (("after_conv1", (96, 55)), ("after_conv2", (256, 27))):
        xl = torch.randn((net.batch, H, H, C), device=dev, generator=gen).relu_().to(dt_t)
        dyl = torch.randn((net.batch, H, H, C), device=dev, generator=gen).to(dt_t)
        yl, dxl = torch.empty_like(xl), torch.empty_like(xl)
        res = {}
        for kind, fn, nb in (("fwd", lambda: singa.lrn_fwd(xl, 5, 1e-4, 0.75, 1.0, out=yl), 2 * es),
                             ("bwd", lambda: singa.lrn_bwd(xl, dyl, 5, 1e-4, 0.75, 1.0, out=dxl), 3 * es)):
            for _ in range(3):
                fn()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(20):
                fn()
            e1.record()
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / 20
            gbs = xl.numel() * nb / (ms / 1e3) / 1e9
            res[kind] = {"ms": round(ms, 4), "GB_per_s": round(gbs, 1), "frac_hbm_peak": round(gbs / PEAK["hbm_gbs"], 4)}
        lrn[name] = dict(res, shape=[net.batch, C, H, H])
        del xl, dyl, yl, dxl

    return lrn


def cpu_baseline(w, n_images, need_input_grad=False):
    """The oracle (fp64 C, OpenMP) on a bounded sample of the same step: the
    full forward/backward of `n_images` images of the workload plus the
    update of all parameters."""
    import numpy as np
    import oracle
    from oracle import net as onet
    from paper_1603_07846_amd import workloads as wl

    inp = wl.make_inputs(w, batch=n_images)
    params = [(wl.round_bf16(p.w) if w.dtype == "bf16" else p.w, p.b) for p in inp.params]
    master = [(p.w, p.b) for p in inp.params]
    oracle.conv_out(1, 1, 0, 1)  # load the library outside the timed region
    t0 = time.perf_counter()
    onet.train_one_batch(w.layers, inp.x, params, master=master, labels=inp.labels, dy_top=inp.dy, lr=w.lr,
                         momentum=w.momentum, wd=w.weight_decay, need_input_grad=need_input_grad,
                         store=oracle.round_bf16 if w.dtype == "bf16" else None)
    dt = time.perf_counter() - t0
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    return {"value": n_images / dt, "unit": "images/s", "cores": threads, "kind": "oracle",
            "sample": "%d of %d images through the full step (forward, backward, update of all %d parameters), "
                      "fp64, %.1f s" % (n_images, w.batch, sum(p.w.size + (0 if p.b is None else p.b.size)
                                                            for p in inp.params), dt),
            "seconds": dt, "host_cpus": os.cpu_count()}


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on exactly one GPU: the library has no multi-GPU path "
              "(--gpus %d, WORLD_SIZE %d requested)" % (args.gpus, world), file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_1603_07846_amd import net as gnet
    from paper_1603_07846_amd import singa
    from paper_1603_07846_amd import workloads as wl

    w = wl.WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    inp = wl.make_inputs(w)
    net = gnet.Net(w, device=dev, concurrent_wgrad=not args.single_stream)
    net.load_params(inp.params)
    x = net.to_device_input(inp.x)
    labels = torch.from_numpy(inp.labels).to(dev) if inp.labels is not None else None
    dy = net.to_device_input(inp.dy) if inp.dy is not None else None
    torch.cuda.synchronize()

    for _ in range(args.warmup):
        net.train_one_batch(x, labels=labels, dy_top=dy)
    torch.cuda.synchronize()

    def timed(step):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            step()
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) * 1e3 / args.steps

    def eager_step():
        net.train_one_batch(x, labels=labels, dy_top=dy)

    # timed region: K steps replayed from a HIP graph of one step, and K steps
    # launched eagerly (the step's two streams overlap more when launched
    # eagerly); `value` is the faster of the two
    graph_ms = None
    graph = None
    if not args.eager:
        graph = net.capture(x, labels=labels, dy_top=dy)
        for _ in range(3):
            graph.replay()
        graph_ms = timed(graph.replay)
    eager_ms = timed(eager_step)
    launch = "eager" if graph_ms is None or eager_ms < graph_ms else "hip_graph"
    ms_per_step = eager_ms if launch == "eager" else graph_ms
    loss = float(net.layers[-1].loss[0].item()) if w.classes else None
    images_per_s = net.batch / (ms_per_step / 1e3)

    # per-kernel pass: the same K steps launched eagerly on one stream (each
    # kernel alone on the GPU), every launch bracketed by HIP events
    side = net.wgrad_stream
    net.wgrad_stream = None
    singa.trace_enable(True)
    traced_ms = timed(eager_step)
    singa.trace_enable(False)
    net.wgrad_stream = side
    recs = singa.trace_records()
    # the graphics clock under the same load (outside every timed region)
    clock = GfxClock()
    if not args.steps_only:
        clock.steady(eager_step)

    # per-kernel aggregates over the timed steps
    agg = {}
    for name, ms, work, unit in recs:
        a = agg.setdefault(name, {"launches": 0, "ms": 0.0, "work": 0.0, "unit": unit})
        a["launches"] += 1
        a["ms"] += ms
        a["work"] += work
    conv_flops = sum(a["work"] for n, a in agg.items() if is_conv_kernel(n))
    conv_ms = sum(a["ms"] for n, a in agg.items() if is_conv_kernel(n) or is_conv_helper(n))
    is_bf16 = w.dtype == "bf16"
    mfma_peak = PEAK["bf16_tflops"] if is_bf16 else PEAK["f32_tflops"]
    conv_tflops = conv_flops / (conv_ms / 1e3) / 1e12 if conv_ms > 0 else 0.0
    kernel_ms = sum(a["ms"] for a in agg.values())

    dom_name, dom = max(agg.items(), key=lambda kv: kv[1]["ms"])
    avg_ms = dom["ms"] / dom["launches"]
    per_launch = dom["work"] / dom["launches"]
    if dom["unit"] == "flop":
        achieved = per_launch / (avg_ms / 1e3) / 1e12
        peak = mfma_peak  # the kernels compute in the workload's dtype
        roof = {"bound": "mfma", "unit": "TFLOP/s"}
    else:
        achieved = per_launch / (avg_ms / 1e3) / 1e9
        peak = PEAK["hbm_gbs"]
        roof = {"bound": "hbm", "unit": "GB/s"}
    roof.update({"kernel": dom_name, "achieved": round(achieved, 2), "peak": peak,
                 "frac": round(achieved / peak, 4), "traffic": measured_traffic(dom_name),
                 "avg_launch_ms": round(avg_ms, 4), "work_per_launch": per_launch,
                 "launches_per_step": dom["launches"] / args.steps})
    # the MFMA peak scales with the graphics clock: the same fraction priced
    # at the clock measured under the same steps
    mhz = clock.mhz()
    if roof["bound"] == "mfma" and mhz:
        roof["peak_at_measured_sclk"] = round(peak * mhz / GfxClock.NOMINAL_MHZ, 1)
        roof["frac_at_measured_sclk"] = round(achieved / roof["peak_at_measured_sclk"], 4)

    upd = agg.get("sgd_kernel")
    update = None
    if upd:
        gbs = upd["work"] / (upd["ms"] / 1e3) / 1e9
        update = {"ms_per_step": round(upd["ms"] / args.steps, 4), "GB_per_s": round(gbs, 1),
                  "frac_hbm_peak": round(gbs / PEAK["hbm_gbs"], 4), "bytes_per_param": 22 if is_bf16 else 20,
                  "params_per_step": int(upd["work"] / args.steps / (22 if is_bf16 else 20)),
                  "note": "layers whose update is not fused into their filter-gradient kernel"}
    updaters = lrn = None
    if not args.steps_only:
        updaters = measure_updaters(net, w)
        lrn = measure_lrn(net, dev, is_bf16)

    kernels = sorted(({"kernel": n, "launches_per_step": a["launches"] / args.steps,
                       "ms_per_step": round(a["ms"] / args.steps, 4),
                       ("TFLOP/s" if a["unit"] == "flop" else "GB/s"):
                           round(a["work"] / (a["ms"] / 1e3) / (1e12 if a["unit"] == "flop" else 1e9), 2)}
                      for n, a in agg.items()), key=lambda d: -d["ms_per_step"])

    out = {
        "metric": METRIC,
        "value": round(images_per_s, 2),
        "unit": "images/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if is_bf16 else "f32",
        "data": "synthetic",
        "config": {"workload": {5: "alexnet_shaped_train_step", 6: "alexnet_lrn_train_step"}.get(
                       args.workload, "workload%d" % args.workload),
                   "description": w.name, "global_batch": net.batch, "image": list(w.in_shape),
                   "classes": w.classes, "params": net.n_params, "layout": "NHWC",
                   "parallelism": "none (1 GPU)"},
        "conv_fwd_bwd_tflops": round(conv_tflops, 2),
        "conv_frac_mfma_peak": round(conv_tflops / mfma_peak, 4),
        "conv_frac_mfma_peak_at_measured_sclk": (round(conv_tflops / (mfma_peak * mhz / GfxClock.NOMINAL_MHZ), 4)
                                                 if mhz else None),
        "sclk": clock.summary(),
        "conv_gflop_per_step": round(conv_flops / args.steps / 1e9, 2),
        "conv_ms_per_step": round(conv_ms / args.steps, 4),
        "kernel_ms_per_step": round(kernel_ms / args.steps, 4),
        "launch": launch,
        "graph_ms_per_step": None if graph_ms is None else round(graph_ms, 4),
        "eager_ms_per_step": round(eager_ms, 4),
        "traced_eager_ms_per_step": round(traced_ms, 4),
        "loss": loss,
        "roofline": roof,
        "update": update,
        "updaters_full_buffer": updaters,
        "lrn_alone": lrn,
        "kernels": kernels[:16],
    }
    out["conv_gflop_per_step_algorithmic"] = round(step_conv_flops(w, net.batch) / 1e9, 2)
    if not args.no_configs and not args.steps_only and args.workload in (5, 6):
        graph = None
        del net, x, labels, dy
        torch.cuda.empty_cache()
        out["configs"] = {str(i): measure_config(i, args.steps, args.warmup) for i in (1, 2, 3, 4)}
        if not args.no_cpu_baseline:
            # the oracle on a bounded sample of each of them (a few seconds in all)
            for i, n_img in CONFIG_CPU_IMAGES.items():
                c = out["configs"][str(i)]
                c["cpu_baseline"] = cpu_baseline(wl.WORKLOADS[i], n_img, need_input_grad=i == 1)
                c["speedup_vs_oracle"] = round(c["images_per_s"] / c["cpu_baseline"]["value"], 1)
    if not args.no_cpu_baseline and not args.steps_only:
        out["cpu_baseline"] = cpu_baseline(w, args.cpu_images)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

#!/usr/bin/env python3
"""Benchmark of the QUAN hot path on one MI355X.

One step = one pass of the whole hot path over one batch of a workload: for
every layer, pack the four real kernels, then the quaternion (Hamilton)
convolution with IQBN (+ReLU where the layer has it) behind it
(quan_qconv2d_iqbn_forward with the library's default statistics mode: a
separate IQBN pass after the plain convolution where the tensor takes the
one-launch or the merged two-launch form, else per-tile statistics in the
convolution's epilogue), through libquan's C ABI
on torch's current stream.  Inputs are seeded synthetic tensors already
resident in HBM when the timed region starts.  The same steps are then timed
with each statistics mode forced (epilogue, separate pass) and in inference
form (stored statistics folded into the convolution's epilogue), and run
with every kernel on its own (pack, convolution, IQBN) for per-kernel times;
the Poincare input mapping is timed on an ImageNet-sized batch.

Prints ONE JSON line:
  value        useful convolution TFLOP/s over whole steps (pack + conv + IQBN);
               useful FLOPs = 2 * N*Ho*Wo * 4Cout * 4Cin * k^2 per layer
  qconv2d      the convolution kernel alone: TFLOP/s and fraction of the bf16
               dense MFMA peak (2516.6 TFLOP/s)
  iqbn         the stand-alone IQBN: GB/s of algorithmic traffic (two reads +
               one write of the tensor) and fraction of 8 TB/s, cold (input
               evicted from the caches first; the headline) and warm (input
               just written by the convolution)
  other_configs  the same figures for the detection pair (3x3 s2 + 1x1) and
               the deep stack (four 256 -> 256 blocks): fused step, per-layer
               convolution TFLOP/s and share of the MFMA peak, IQBN cold/warm
  roofline     the dominant kernel (the convolution) against its roofline,
               timed with HIP events on the stream it runs on
  cpu_baseline the CPU oracle timed on a bounded sample of the same workload
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

MFMA_PEAK_TFLOPS = {"bf16": 2516.6, "fp32": 157.3}
HBM_PEAK_GBPS = 8000.0
METRIC = "qconv2d bf16 TFLOP/s + % MFMA peak; IQBN GB/s + % HBM peak"
DEFAULT_WORKLOAD = "imagenet_stage"
# the other configurations the targets apply to, reported as sub-records
OTHER_CONFIGS = ["detection_pair", "deep_stack"]
# HBM bytes per step of the convolution kernel (all layers of the workload),
# from rocprofv3 --pmc FETCH_SIZE and WRITE_SIZE runs of this benchmark, each
# scaled by what the same counter reads for a 512 MiB device copy (FETCH x2.0,
# WRITE x1.0); the runs are summarised in profiles/qconv2d_<workload>_hbm.md.
# A figure is reported only while the kernel sources are the ones it was
# measured on (sha256 prefix of the convolution sources, concatenated).
CONV_TRAFFIC = {
    "imagenet_stage": {"bytes": 219183469, "kernel_sha256": "1cfe60a151dc3a89"},
    "detection_pair": {"bytes": 276743986, "kernel_sha256": "1cfe60a151dc3a89"},
    "deep_stack": {"bytes": 260089274, "kernel_sha256": "1cfe60a151dc3a89"},
}
CONV_SOURCES = [os.path.join(ROOT, "paper_2509_05512_amd", "csrc", f)
                for f in ("qconv2d_gfx950.hip", "qconv2d_pointwise_gfx950.hip", "gfx950_dma.h")]


def conv_source_sha():
    """sha256 prefix of the convolution kernels' sources, concatenated."""
    import hashlib
    h = hashlib.sha256()
    for path in CONV_SOURCES:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def conv_traffic(workload):
    entry = CONV_TRAFFIC.get(workload)
    if entry is None:
        return None
    return entry["bytes"] if conv_source_sha() == entry["kernel_sha256"] else None


def parse_args():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    # a few steps leave the GPU still raising its clocks (measured: 5 warmup
    # steps 788-819 TFLOP/s, 50 steps 870-882 on the same box); 50 steps of
    # this workload take ~15 ms
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--no-other-configs", action="store_true",
                    help="measure only --workload (profiling runs)")
    ap.add_argument("--no-cpu-baseline", action="store_true",
                    help="skip the CPU oracle leg (profiling runs)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target duration of the CPU oracle sample")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run device-to-device copies of MIB MiB (calibrates the HBM "
                         "byte counters against a transfer of known size) and exit")
    return ap.parse_args()


def copy_calibration(mib, reps=5):
    """Copies of a known size, for scaling FETCH_SIZE / WRITE_SIZE."""
    import torch
    n = mib * (1 << 20) // 2
    src = torch.ones(n, dtype=torch.bfloat16, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes_per_dispatch": n * 2, "dispatches": reps}), flush=True)


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def build_layers(wl, tens, dev, quan, torch):
    """Device tensors and preallocated outputs for every layer."""
    layers = []
    n, h, w = wl.n, wl.h, wl.w
    x = quan.to_device_layout(tens.x.to(dev))
    for L, lt, d in zip(wl.layers, tens.layers, wl.layer_dims()):
        ws = [lt.weight[q].contiguous().to(dev) for q in range(4)]
        layer = dict(
            spec=L, dims=d, x=x, w=ws,
            bias=lt.bias.contiguous().to(dev) if lt.bias is not None else None,
            gamma=lt.gamma.to(dev), beta=lt.beta.to(dev),
            packed=torch.empty(quan.quan_qconv2d_packed_bytes(L.c_in, L.c_out, L.k, L.k, x.dtype),
                               dtype=torch.uint8, device=dev),
            y=quan.empty_qmap(n, L.c_out, d["ho"], d["wo"], x.dtype, dev),
            z=quan.empty_qmap(n, L.c_out, d["ho"], d["wo"], x.dtype, dev),
            mean=torch.empty(4, L.c_out, device=dev), var=torch.empty(4, L.c_out, device=dev),
        )
        layers.append(layer)
        x = layer["z"]
    return layers


def run_step_fused(layers, quan, eps=1e-5, stats="auto"):
    """One step of the hot path as a caller runs it: per layer, pack the
    kernels, then the convolution with IQBN (+ ReLU) behind it."""
    for ly in layers:
        L = ly["spec"]
        quan.quan_qconv2d_pack_weights(*ly["w"], packed=ly["packed"])
        quan.quan_qconv2d_iqbn_forward(ly["x"], ly["packed"], (L.c_out, L.c_in, L.k, L.k),
                                       ly["gamma"], ly["beta"], bias=ly["bias"], stride=L.stride,
                                       pad=L.pad, dilation=L.dilation, eps=eps, relu=L.relu,
                                       out=ly["z"], mean=ly["mean"], var=ly["var"], stats=stats)


def run_step_inference(layers, quan, eps=1e-5):
    """The step in inference form: per layer, pack the kernels, then the
    convolution with IQBN (+ ReLU) folded into its epilogue, using the
    statistics the last training-form step produced as stored statistics."""
    for ly in layers:
        L = ly["spec"]
        quan.quan_qconv2d_pack_weights(*ly["w"], packed=ly["packed"])
        quan.quan_qconv2d_iqbn_inference(ly["x"], ly["packed"], (L.c_out, L.c_in, L.k, L.k), ly["mean"],
                                         ly["var"], ly["gamma"], ly["beta"], bias=ly["bias"],
                                         stride=L.stride, pad=L.pad, dilation=L.dilation, eps=eps,
                                         relu=L.relu, out=ly["z"])


def time_separable(layers, quan, steps):
    """The separable convolution (eq. 7) on every layer's packed weights:
    microseconds per step (all layers) of the convolution alone."""
    import torch
    def once():
        for ly in layers:
            L = ly["spec"]
            quan.quan_qconv2d_separable_forward_packed(ly["x"], ly["packed"], (L.c_out, L.c_in, L.k, L.k),
                                                       bias=ly["bias"], stride=L.stride, pad=L.pad,
                                                       dilation=L.dilation, out=ly["y"])
    for _ in range(2):
        once()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for _ in range(steps):
        once()
    end.record()
    torch.cuda.synchronize()
    return start.elapsed_time(end) * 1e3 / steps


def time_separable_backward(layers, quan, steps):
    """The separable form's gradients (eqs. 8-10) of every layer for a seeded
    dL/dy: microseconds per step of the input gradient and of the weight +
    bias gradients."""
    import torch
    g = torch.Generator(device="cpu").manual_seed(7)
    grads = [quan.to_device_layout(torch.randn(tuple(ly["y"].shape), generator=g).to(ly["y"].dtype)
                                   .to(ly["y"].device)) for ly in layers]
    # events of every step, one synchronisation at the end: the host queues
    # ahead, so no interval holds the host's own dispatch time
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps + 1)]

    def once(e):
        e[0].record()
        for ly, dy in zip(layers, grads):
            L = ly["spec"]
            quan.quan_qconv2d_separable_backward_data(dy, *ly["w"], (ly["x"].shape[3], ly["x"].shape[4]),
                                                      stride=L.stride, pad=L.pad, dilation=L.dilation)
        e[1].record()
        for ly, dy in zip(layers, grads):
            L = ly["spec"]
            quan.quan_qconv2d_separable_backward_weight(ly["x"], dy, (L.k, L.k), stride=L.stride, pad=L.pad,
                                                        dilation=L.dilation)
        e[2].record()
    once(evs[0])
    torch.cuda.synchronize()
    for s in range(steps):
        once(evs[s + 1])
    torch.cuda.synchronize()
    tot = [sum(e[0].elapsed_time(e[1]) for e in evs[1:]) * 1e3, sum(e[1].elapsed_time(e[2]) for e in evs[1:]) * 1e3]
    return [t / steps for t in tot]


def time_iqbn_cold(layers, quan, steps, eps):
    """The stand-alone IQBN of each layer with its input evicted from the
    caches first: before each timed rep a 512 MiB buffer is read (twice the
    256 MB Infinity Cache; a read leaves no dirty lines whose write-back would
    land inside the timed region).  Median microseconds per layer."""
    import torch
    dev = layers[0]["y"].device
    flush_buf = torch.zeros(128 * 2**20, dtype=torch.float32, device=dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    med = []
    for ly in layers:
        fn = quan.quan_iqbn_relu_forward if ly["spec"].relu else quan.quan_iqbn_forward
        times = []
        for _ in range(max(steps, 5)):
            flush_buf.sum()
            e0.record()
            fn(ly["y"], ly["gamma"], ly["beta"], eps, out=ly["z"], mean=ly["mean"], var=ly["var"])
            e1.record()
            torch.cuda.synchronize()
            times.append(e0.elapsed_time(e1) * 1e3)
        times.sort()
        med.append(times[len(times) // 2])
    del flush_buf
    return med


def time_backward(layers, quan, steps, eps):
    """The backward pass of every layer, last layer first: IQBN's gradient,
    then the convolution's input and weight (+ bias) gradients, for a seeded
    dL/dz.  Microseconds per step of each part."""
    import torch
    g = torch.Generator(device="cpu").manual_seed(6)
    grads = [quan.to_device_layout(torch.randn(tuple(ly["z"].shape), generator=g).to(ly["z"].dtype)
                                   .to(ly["z"].device)) for ly in layers]
    # events of every step, one synchronisation at the end: the host queues
    # ahead, so no interval holds the host's own dispatch time
    evs = [[[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in layers] for _ in range(steps + 1)]

    def once(step_evs):
        for li in reversed(range(len(layers))):
            ly, L = layers[li], layers[li]["spec"]
            ev = step_evs[li]
            ev[0].record()
            dy, _, _ = quan.quan_iqbn_backward(ly["y"], grads[li], ly["mean"], ly["var"], ly["gamma"],
                                               y=ly["z"] if L.relu else None, eps=eps)
            ev[1].record()
            quan.quan_qconv2d_backward_data(dy, *ly["w"], (ly["x"].shape[3], ly["x"].shape[4]), stride=L.stride,
                                            pad=L.pad, dilation=L.dilation)
            ev[2].record()
            quan.quan_qconv2d_backward_weight(ly["x"], dy, (L.k, L.k), stride=L.stride, pad=L.pad,
                                              dilation=L.dilation)
            ev[3].record()
    once(evs[0])
    torch.cuda.synchronize()
    for s in range(steps):
        once(evs[s + 1])
    torch.cuda.synchronize()
    tot = [0.0, 0.0, 0.0]
    for step_evs in evs[1:]:
        for ev in step_evs:
            for i in range(3):
                tot[i] += ev[i].elapsed_time(ev[i + 1]) * 1e3
    return [t / steps for t in tot]


def time_poincare(quan, steps, dev):
    """The Poincare input mapping of one ImageNet-sized bf16 batch
    (64 x 3 x 224 x 224): microseconds per launch and algorithmic GB/s
    (3 reads + 4 writes of a 2-byte element per pixel); and a stem
    convolution on it with the map fused into its loads against the two
    separate passes."""
    import torch
    n, h, w = 64, 224, 224
    g = torch.Generator(device="cpu").manual_seed(5)
    rgb = torch.rand((n, 3, h, w), generator=g).to(torch.bfloat16).to(dev)
    q = quan.quan_poincare_map(rgb)
    for _ in range(3):
        quan.quan_poincare_map(rgb, out=q)
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for _ in range(steps):
        quan.quan_poincare_map(rgb, out=q)
    end.record()
    torch.cuda.synchronize()
    us = start.elapsed_time(end) * 1e3 / steps
    gbps = n * h * w * 7 * 2 / (us * 1e-6) / 1e9
    # the stem convolution on the mapped batch (3x3, stride 2, pad 1, 16
    # quaternion channels): the map fused into the convolution's loads,
    # against the map followed by the convolution
    c_out, k = 16, 3
    w = [(torch.randn((c_out, 1, k, k), generator=g) / 6.0).to(torch.bfloat16).to(dev) for _ in range(4)]
    packed = quan.quan_qconv2d_pack_weights(*w)
    shape = (c_out, 1, k, k)
    y = quan.quan_qconv2d_poincare_forward(rgb, packed, shape, stride=2, pad=1)

    def fused():
        quan.quan_qconv2d_poincare_forward(rgb, packed, shape, stride=2, pad=1, out=y)

    def two_pass():
        quan.quan_poincare_map(rgb, out=q)
        quan.quan_qconv2d_forward_packed(q, packed, shape, stride=2, pad=1, out=y)

    times = {}
    for name, fn in (("fused", fused), ("two_pass", two_pass), ("fused2", fused), ("two_pass2", two_pass)):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        start.record()
        for _ in range(steps):
            fn()
        end.record()
        torch.cuda.synchronize()
        times[name] = start.elapsed_time(end) * 1e3 / steps
    stem_flops = 2 * n * y.shape[3] * y.shape[4] * 4 * c_out * 4 * 1 * k * k
    fused_us = min(times["fused"], times["fused2"])
    return {"workload": "64x3x224x224 bf16", "us": round(us, 3), "gbps": round(gbps, 1),
            "frac_hbm_peak": round(gbps / HBM_PEAK_GBPS, 4),
            "stem": {"conv": "3x3 stride 2 pad 1, 1 -> 16 quaternion channels",
                     "fused_us": round(fused_us, 3),
                     "two_pass_us": round(min(times["two_pass"], times["two_pass2"]), 3),
                     "fused_tflops": round(stem_flops / (fused_us * 1e-6) / 1e12, 2)}}


def run_step(layers, quan, events=None, eps=1e-5):
    """The same step with every kernel on its own (pack, convolution, the
    three IQBN passes), events between them: per-kernel times."""
    for li, ly in enumerate(layers):
        L = ly["spec"]
        if events is not None:
            events[li][0].record()
        quan.quan_qconv2d_pack_weights(*ly["w"], packed=ly["packed"])
        if events is not None:
            events[li][1].record()
        quan.quan_qconv2d_forward_packed(ly["x"], ly["packed"], (L.c_out, L.c_in, L.k, L.k),
                                         bias=ly["bias"], stride=L.stride, pad=L.pad,
                                         dilation=L.dilation, out=ly["y"])
        if events is not None:
            events[li][2].record()
        fn = quan.quan_iqbn_relu_forward if L.relu else quan.quan_iqbn_forward
        fn(ly["y"], ly["gamma"], ly["beta"], eps, out=ly["z"], mean=ly["mean"], var=ly["var"])
        if events is not None:
            events[li][3].record()


def per_kernel_times(layers, quan, steps, eps):
    """Milliseconds per layer of the pack, the convolution and the three IQBN
    passes, each launch on its own with HIP events between them on torch's
    current stream (the stream the kernels run on), averaged over steps."""
    import torch
    for _ in range(2):
        run_step(layers, quan, eps=eps)
    events = [[[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in layers] for _ in range(steps)]
    torch.cuda.synchronize()
    for s in range(steps):
        run_step(layers, quan, events=events[s], eps=eps)
    torch.cuda.synchronize()
    def avg(li, a, b):
        return sum(events[s][li][a].elapsed_time(events[s][li][b]) for s in range(steps)) / steps
    return ([avg(li, 0, 1) for li in range(len(layers))], [avg(li, 1, 2) for li in range(len(layers))],
            [avg(li, 2, 3) for li in range(len(layers))])


def time_fused_steps(layers, quan, steps, eps, stats="auto"):
    """Milliseconds per whole fused step (every layer: pack, convolution with
    IQBN), HIP events around `steps` back-to-back steps."""
    import torch
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for _ in range(steps):
        run_step_fused(layers, quan, eps=eps, stats=stats)
    end.record()
    torch.cuda.synchronize()
    return start.elapsed_time(end) / steps


# Targets the measurement is held to: the convolution at >= 50% of the bf16
# MFMA peak, IQBN at >= 70% of HBM bandwidth.  The detection pair (3x3 s2 +
# 1x1) is judged as a pair: 73.8 GFLOP at 50% of 2516.6 TFLOP/s = 58.7 us.
def layer_records(wl, dims, conv_ms, iqbn_ms, cold_us, pack_ms=None):
    esz = 2 if wl.dtype == "bf16" else 4
    peak = MFMA_PEAK_TFLOPS[wl.dtype]
    recs = []
    for li, L in enumerate(wl.layers):
        d = dims[li]
        nbytes = 3 * wl.n * d["ho"] * d["wo"] * 4 * L.c_out * esz
        tf = d["useful_flops"] / (conv_ms[li] * 1e-3) / 1e12
        r = {"layer": li, "c_in": L.c_in, "c_out": L.c_out, "k": L.k, "stride": L.stride, "pad": L.pad,
             "h_out": d["ho"], "w_out": d["wo"]}
        if pack_ms is not None:
            r["pack_us"] = round(pack_ms[li] * 1e3, 3)
        # the least HBM traffic of the layer: its input and output once, the
        # four kernels once
        conv_bytes = (wl.n * d["h"] * d["w"] * 4 * L.c_in + wl.n * d["ho"] * d["wo"] * 4 * L.c_out
                      + 4 * L.c_out * L.c_in * L.k * L.k) * esz
        conv_gbps = conv_bytes / (conv_ms[li] * 1e-3) / 1e9
        r.update({
            "qconv2d_us": round(conv_ms[li] * 1e3, 3), "qconv2d_tflops": round(tf, 2),
            "qconv2d_frac_mfma_peak": round(tf / peak, 4),
            "qconv2d_algorithmic_gbps": round(conv_gbps, 1),
            "qconv2d_frac_hbm_peak": round(conv_gbps / HBM_PEAK_GBPS, 4),
            "iqbn_cold_us": round(cold_us[li], 3),
            "iqbn_cold_gbps": round(nbytes / (cold_us[li] * 1e-6) / 1e9, 1),
            "iqbn_cold_frac_hbm_peak": round(nbytes / (cold_us[li] * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
            "iqbn_warm_us": round(iqbn_ms[li] * 1e3, 3),
            "iqbn_warm_gbps": round(nbytes / (iqbn_ms[li] * 1e-3) / 1e9, 1),
        })
        recs.append(r)
    return recs


def measure_config(name, args, dev, quan, workloads):
    """A sub-record for another target configuration: the fused step, and per
    layer the convolution alone and IQBN cold and warm."""
    import torch
    wl = workloads.WORKLOADS[name]
    log(f"[bench] config {wl.name}: {wl.description}")
    tens = workloads.generate(wl)
    layers = build_layers(wl, tens, dev, quan, torch)
    for _ in range(args.warmup):
        run_step_fused(layers, quan, eps=wl.eps)
    step_ms = time_fused_steps(layers, quan, args.steps, wl.eps)
    _, conv_ms, iqbn_ms = per_kernel_times(layers, quan, args.steps, wl.eps)
    cold_us = time_iqbn_cold(layers, quan, args.steps, wl.eps)
    dims = wl.layer_dims()
    flops = sum(d["useful_flops"] for d in dims)
    peak = MFMA_PEAK_TFLOPS[wl.dtype]
    esz = 2 if wl.dtype == "bf16" else 4
    nbytes = sum(3 * wl.n * d["ho"] * d["wo"] * 4 * L.c_out * esz for d, L in zip(dims, wl.layers))
    conv_tf = flops / (sum(conv_ms) * 1e-3) / 1e12
    rec = {
        "workload": wl.name, "description": wl.description,
        "useful_gflop_per_step": round(flops / 1e9, 3),
        "step_us": round(step_ms * 1e3, 3),
        "step_tflops": round(flops / (step_ms * 1e-3) / 1e12, 2),
        "qconv2d": {"us_per_step": round(sum(conv_ms) * 1e3, 3), "tflops": round(conv_tf, 2),
                    "frac_mfma_peak": round(conv_tf / peak, 4),
                    # HBM bytes per step of the convolution launches (profiles/), or None
                    "traffic": conv_traffic(name)},
        "iqbn": {"cold_us_per_step": round(sum(cold_us), 3),
                 "cold_gbps": round(nbytes / (sum(cold_us) * 1e-6) / 1e9, 1),
                 "cold_frac_hbm_peak": round(nbytes / (sum(cold_us) * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
                 "warm_us_per_step": round(sum(iqbn_ms) * 1e3, 3),
                 "warm_gbps": round(nbytes / (sum(iqbn_ms) * 1e-3) / 1e9, 1)},
        "per_layer": layer_records(wl, dims, conv_ms, iqbn_ms, cold_us),
    }
    if wl.name == "detection_pair":
        rec["pair_conv_us"] = round(sum(conv_ms) * 1e3, 3)
        rec["pair_conv_target_us"] = round(flops / (0.5 * peak * 1e12) * 1e6, 1)
    for r in rec["per_layer"]:
        log(f"[bench] {wl.name} layer {r}")
    del layers
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return rec


def cpu_model():
    """The host CPU's model name, as lscpu reports it."""
    import subprocess
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.startswith("Model name:"):
                return line.split(":", 1)[1].strip()
    except (OSError, subprocess.SubprocessError):
        pass
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(wl, tens, target_s):
    """The oracle on the first images of the batch (all layers, conv + IQBN),
    timed on this host's cores.  Returns the oracle's useful-FLOP rate."""
    import numpy as np
    import oracle
    import torch

    def run(n_img):
        x = tens.x[:n_img].to(torch.float64).numpy()
        flops = 0
        t0 = time.perf_counter()
        for L, lt in zip(wl.layers, tens.layers):
            w = lt.weight.to(torch.float64).numpy()
            b = lt.bias.to(torch.float64).numpy() if lt.bias is not None else None
            y = oracle.qconv2d(x, w, b, L.stride, L.pad, L.dilation)
            flops += 2 * y.shape[0] * y.shape[3] * y.shape[4] * 4 * L.c_out * 4 * L.c_in * L.k * L.k
            x, _, _ = oracle.iqbn(y, lt.gamma.double().numpy(), lt.beta.double().numpy(),
                                  wl.eps, L.relu)
        return time.perf_counter() - t0, flops

    oracle.default()  # build/load outside the timed region
    t1, f1 = run(1)
    n_img = int(max(1, min(wl.n, round(target_s / max(t1, 1e-6)))))
    if n_img > 1:
        t, f = run(n_img)
    else:
        t, f = t1, f1
    threads = int(os.environ.get("OMP_NUM_THREADS", "0") or 0) or len(os.sched_getaffinity(0))
    return {
        "value": f / t / 1e12,
        "unit": "TFLOP/s",
        "cores": threads,
        "cpu_model": cpu_model(),
        "kind": "oracle",
        "sample": f"first {n_img} of {wl.n} images through every layer (conv + IQBN), fp64, "
                  f"{t:.1f} s, {f / 1e9:.2f} GFLOP",
    }


def main():
    args = parse_args()
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on exactly one GPU: the QUAN hot path here is the single-GPU "
              "kernel pair (quaternion conv + IQBN); multi-GPU data parallelism (one all-reduce "
              "of IQBN statistics per layer) is not built.  Use --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2509_05512_amd import quan, workloads

    quan.load_library()  # fails loudly if the HIP library is missing
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    wl = workloads.WORKLOADS[args.workload]
    log(f"[bench] workload {wl.name}: {wl.description}")
    tens = workloads.generate(wl)
    layers = build_layers(wl, tens, dev, quan, torch)
    torch.cuda.synchronize()

    dims = wl.layer_dims()
    conv_flops = [d["useful_flops"] for d in dims]
    esz = 2 if wl.dtype == "bf16" else 4
    iqbn_bytes = [3 * wl.n * d["ho"] * d["wo"] * 4 * L.c_out * esz for d, L in zip(dims, wl.layers)]

    for _ in range(args.warmup):
        run_step_fused(layers, quan, eps=wl.eps)
    torch.cuda.synchronize()
    log(f"[bench] warmup {args.warmup} done; timing {args.steps} steps")

    # the timed region: K whole steps (pack + convolution + IQBN)
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_wall0 = time.perf_counter()
    start.record()
    for s in range(args.steps):
        run_step_fused(layers, quan, eps=wl.eps)
    end.record()
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall0
    total_ms = start.elapsed_time(end)
    ms_per_step = total_ms / args.steps

    # the same steps with each statistics mode forced
    mode_ms = {}
    for mode in ("epilogue", "pass"):
        for _ in range(2):
            run_step_fused(layers, quan, eps=wl.eps, stats=mode)
        torch.cuda.synchronize()
        start.record()
        for s in range(args.steps):
            run_step_fused(layers, quan, eps=wl.eps, stats=mode)
        end.record()
        torch.cuda.synchronize()
        mode_ms[mode] = start.elapsed_time(end) / args.steps
    pass_ms = mode_ms["pass"]

    # the step in inference form (stored statistics folded into the conv)
    for _ in range(2):
        run_step_inference(layers, quan, eps=wl.eps)
    torch.cuda.synchronize()
    start.record()
    for s in range(args.steps):
        run_step_inference(layers, quan, eps=wl.eps)
    end.record()
    torch.cuda.synchronize()
    inference_ms = start.elapsed_time(end) / args.steps
    poincare = time_poincare(quan, args.steps, dev)
    separable_us = time_separable(layers, quan, args.steps)
    sep_bwd_data_us, sep_bwd_weight_us = time_separable_backward(layers, quan, args.steps)
    # the separate-kernel forward leaves y (conv), z (IQBN) and the statistics
    run_step(layers, quan, eps=wl.eps)
    bwd_iqbn_us, bwd_data_us, bwd_weight_us = time_backward(layers, quan, args.steps, wl.eps)

    # per-kernel times: the same steps with every kernel on its own
    pack_ms, conv_ms, iqbn_ms = per_kernel_times(layers, quan, args.steps, wl.eps)
    log(f"[bench] {args.steps} steps: {ms_per_step:.4f} ms/step (wall {1e3 * t_wall / args.steps:.4f})")

    step_flops = sum(conv_flops)
    value = step_flops / (ms_per_step * 1e-3) / 1e12
    conv_tflops = step_flops / (sum(conv_ms) * 1e-3) / 1e12
    peak = MFMA_PEAK_TFLOPS[wl.dtype]
    iqbn_gbps = sum(iqbn_bytes) / (sum(iqbn_ms) * 1e-3) / 1e9
    cold_us = time_iqbn_cold(layers, quan, args.steps, wl.eps)
    iqbn_cold_us = sum(cold_us)
    iqbn_cold_gbps = sum(iqbn_bytes) / (iqbn_cold_us * 1e-6) / 1e9
    per_layer = layer_records(wl, dims, conv_ms, iqbn_ms, cold_us, pack_ms)
    for pl in per_layer:
        log(f"[bench] layer {pl}")
    others = {}
    if not args.no_other_configs:
        for name in OTHER_CONFIGS:
            if name != wl.name:
                others[name] = measure_config(name, args, dev, quan, workloads)

    traffic = conv_traffic(wl.name)
    result = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic",
        "config": {
            "workload": wl.name, "description": wl.description, "batch": wl.n,
            "height": wl.h, "width": wl.w,
            "layers": [{"c_in": L.c_in, "c_out": L.c_out, "k": L.k, "stride": L.stride,
                        "pad": L.pad, "iqbn_relu": L.relu} for L in wl.layers],
            "useful_gflop_per_step": round(step_flops / 1e9, 3),
        },
        "step": "per layer: pack the four kernels, then quan_qconv2d_iqbn_forward with "
                "QUAN_STATS_AUTO (the plain convolution and then IQBN in one launch where "
                "the tensor takes it and holds at least 64 MiB, or in two launches with the "
                "finalize merged into the normalization on tensors of up to 32 MiB with wide "
                "rows; else IQBN statistics in the convolution's epilogue)",
        "stats_epilogue_us_per_step": round(mode_ms["epilogue"] * 1e3, 3),
        "stats_pass_us_per_step": round(pass_ms * 1e3, 3),
        "inference_us_per_step": round(inference_ms * 1e3, 3),
        "inference_tflops": round(step_flops / (inference_ms * 1e-3) / 1e12, 2),
        "poincare": poincare,
        "backward": {
            # per step (all layers): IQBN gradient, conv input gradient,
            # conv weight + bias gradients; useful FLOPs of each conv
            # gradient equal the forward's
            "iqbn_us": round(bwd_iqbn_us, 3),
            "data_us": round(bwd_data_us, 3),
            "data_tflops": round(step_flops / (bwd_data_us * 1e-6) / 1e12, 2),
            "weight_us": round(bwd_weight_us, 3),
            "weight_tflops": round(step_flops / (bwd_weight_us * 1e-6) / 1e12, 2),
        },
        "separable": {
            "us_per_step": round(separable_us, 3),
            # eq. 7 does a quarter of the Hamilton product's multiply-adds
            "tflops": round(step_flops / 4 / (separable_us * 1e-6) / 1e12, 2),
            "frac_mfma_peak": round(step_flops / 4 / (separable_us * 1e-6) / 1e12 / peak, 4),
            # its gradients (eqs. 8-10): the input gradient runs the mixing
            # inside a Hamilton-shaped block product (16 blocks), the weight
            # gradient sixteen component-pair products; useful FLOPs as eq. 7's
            "backward_data_us": round(sep_bwd_data_us, 3),
            "backward_weight_us": round(sep_bwd_weight_us, 3),
        },
        "separate_kernels_us_per_step": round((sum(pack_ms) + sum(conv_ms) + sum(iqbn_ms)) * 1e3, 3),
        "qconv2d": {
            "tflops": round(conv_tflops, 2),
            "frac_mfma_peak": round(conv_tflops / peak, 4),
            "us_per_step": round(sum(conv_ms) * 1e3, 3),
            "pack_us_per_step": round(sum(pack_ms) * 1e3, 3),
        },
        "iqbn": {
            # headline: the tensor evicted from L2 and the Infinity Cache first
            "gbps": round(iqbn_cold_gbps, 1),
            "frac_hbm_peak": round(iqbn_cold_gbps / HBM_PEAK_GBPS, 4),
            "us_per_step": round(iqbn_cold_us, 3),
            # beside it, warm: the tensor just written by the convolution
            "warm_gbps": round(iqbn_gbps, 1),
            "warm_frac_hbm_peak": round(iqbn_gbps / HBM_PEAK_GBPS, 4),
            "warm_us_per_step": round(sum(iqbn_ms) * 1e3, 3),
        },
        "per_layer": per_layer,
        "other_configs": others,
        "roofline": {
            "bound": "mfma",
            "kernel": "qconv2d_igemm",
            "achieved": round(conv_tflops, 2),
            "peak": peak,
            "unit": "TFLOP/s",
            "frac": round(conv_tflops / peak, 4),
            "traffic": traffic,
        },
    }
    if not args.no_cpu_baseline:
        log("[bench] CPU oracle baseline ...")
        result["cpu_baseline"] = cpu_baseline(wl, tens, args.cpu_seconds)
        log(f"[bench] cpu baseline {result['cpu_baseline']}")
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()

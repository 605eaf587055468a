#!/usr/bin/env python3
"""Throughput of the DenseNet conv5 descriptor-pyramid path on one MI355X.

One step is one pass of the whole path over one batch of synthetic input already resident in HBM:
fused pyramid build (resize, centring, padding, stitching) -> conv1..conv5 with ReLU, LRN and pooling
on every stitched plane -> per-scale conv5 windows -> region windows for 2000 boxes per image.
After the timed steps it also times the paper's per-window baseline (every box of one image warped to
227 x 227 and run through the network on its own) and reports it beside the dense time per image, and
the same batch with cross-image packing (the scales of all 16 images stitched together: 88 planes
instead of 96), reported beside the headline, which keeps each image's own planes, and the latency of
one 25-scale pyramid of one image (fp16), launched eagerly and replayed from a captured graph, and
the workloads that give each scale its own plane (480 x 640 at 8 scales in fp16 and fp32, 227 x 227
at 2 scales in fp32), whose planes of different sizes share one launch per layer.  With --ceilings
it also measures what bounds the kernels on the device: a vendor bf16 GEMM and this library's conv2
and conv3 on random and on zero operands, and device copy/fill bandwidth.
The default workload is a batch of 16 images of 768 x 1024, each a 25-scale 2^-0.1 pyramid on
1200 x 1200 planes (96 planes), bf16 storage with fp32 accumulation.

Prints one JSON line: throughput in 25-scale pyramids/s, the roofline of the dominant kernel (its
average duration measured live with events on its own stream during the timed steps), the conv
MFMA utilisation, and the CPU oracle timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "25-scale conv5 pyramids/sec on 1 GPU + conv MFMA util % of peak"
PEAK_TFLOPS = {"bf16": 2500.0, "f16": 2500.0, "f32": 157.3}
PEAK_HBM_GBS = 8000.0
CONV_NAMES = ("conv1", "conv2", "conv3", "conv4", "conv5")


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawTextHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", choices=("batch16", "single"), default="batch16",
                    help="batch16: 16 images, bf16 (default); single: one image, fp16")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-planes", type=int, default=2,
                    help="planes of image 0 the oracle's conv stack runs on for the CPU baseline")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="after the timed steps, run one plain device copy of this many MiB "
                         "(a known-size reference for hardware byte counters)")
    ap.add_argument("--kernels", action="store_true", help="also print the per-kernel breakdown")
    ap.add_argument("--no-per-window", action="store_true",
                    help="skip the per-window baseline (every box warped to 227 x 227 and run alone)")
    ap.add_argument("--no-packed", action="store_true",
                    help="skip the cross-image packed variant (the batch's scales stitched together)")
    ap.add_argument("--no-single", action="store_true",
                    help="skip the single-image latency figures (one 25-scale pyramid, fp16)")
    ap.add_argument("--no-per-scale", action="store_true",
                    help="skip the per-scale-plane workloads (480x640 at 8 scales, 227x227 at 2)")
    ap.add_argument("--ceilings", action="store_true",
                    help="also measure what bounds the kernels on this device: a bf16 GEMM (torch.mm, "
                         "vendor library) and conv2/conv3 of this library on random and on zero "
                         "operands, and device copy/fill bandwidth")
    return ap.parse_args()


def source_digest() -> str:
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_1404_1869_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(name.encode())
            h.update(f.read())
    return h.hexdigest()[:16]


def load_traffic(kernel: str, workload: str, digest: str):
    """Per-launch HBM bytes of `kernel` from the committed counter summary, if taken on this source."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_hbm_traffic.txt")
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                vals[k.strip()] = v.strip()
    if vals.get("source_digest") != digest:
        return None
    try:
        return float(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: this build runs the whole path on a single MI355X and has "
              "no multi-GPU mode (--gpus must be 1)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_1404_1869_amd import configs as C
    from paper_1404_1869_amd import densenet as D
    from paper_1404_1869_amd import synth, workmodel

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    w = C.XGA_25SCALE_B16 if args.workload == "batch16" else C.XGA_25SCALE
    dtn = w.dtypes[0]
    dt = D.DTYPES[dtn]
    n_img = w.n_img
    boxes_per_img = 2000

    # ---- inputs resident in HBM before the timed region
    imgs = torch.from_numpy(synth.images(w.seeds, w.H, w.W)).to(dev)
    weights = [(torch.from_numpy(a).to(dev), torch.from_numpy(b).to(dev)) for a, b in synth.weights(7)]
    packed = D.densenet_pack_weights(weights, dt)
    boxes = torch.from_numpy(np.concatenate([synth.boxes(105 + b, boxes_per_img, w.H, w.W)
                                             for b in range(n_img)])).to(dev)
    box_img = torch.arange(n_img, dtype=torch.int32, device=dev).repeat_interleave(boxes_per_img)
    params = D.params_for(w)
    planes, plan = D.densenet_build_pyramid(imgs, params, dt)
    ppi = len(plan.planes)
    desc = plan.image_descs(n_img)
    net = D.net_params(pool5=False)
    cf = D.ConvFeatures(desc, dt, net, device=dev)
    c5d = list(cf.c5d)
    n_boxes = boxes.shape[0]
    out_desc = torch.empty((n_boxes, 256 * 36), dtype=torch.float32, device=dev)
    out_scale = torch.empty(n_boxes, dtype=torch.int32, device=dev)

    def step():
        D.densenet_build_pyramid(imgs, params, dt, out=planes)
        cf(planes, packed)
        D.densenet_region_windows(cf.conv5, c5d, dt, plan, w.pad, ppi, boxes, box_img, out=out_desc,
                                  scale=out_scale)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # ---- per-kernel breakdown (untimed pass, every launch traced) picks the dominant kernel
    D.profile_start()
    for _ in range(3):
        step()
    torch.cuda.synchronize()
    breakdown = D.profile_stop()
    dominant = max(breakdown, key=lambda k: breakdown[k][1])

    # ---- timed region: K steps, only the dominant kernel bracketed by events on its stream
    D.profile_start([dominant])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    live = D.profile_stop()
    elapsed = t1 - t0
    ms_per_step = 1e3 * elapsed / args.steps
    value = n_img * args.steps / elapsed

    if args.copy_mib > 0:
        src = torch.empty(args.copy_mib << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()

    # ---- algorithmic work per launch (whole planes, MFMA padding not counted)
    n_planes = len(desc)
    PH, PW = plan.planes[0].h, plan.planes[0].w
    fl = workmodel.conv_flops(PH, PW)
    es = 4 if dtn == "f32" else 2
    sd = workmodel.sides(PH)
    work = {f"conv{i + 1}": ("mfma", fl[i] * n_planes) for i in range(5)}
    work["lrn_pool1"] = ("hbm", (sd[0] ** 2 + sd[1] ** 2) * 96 * es * n_planes)
    work["lrn_pool2"] = ("hbm", (sd[2] ** 2 + sd[3] ** 2) * 256 * es * n_planes)
    work["build_planes"] = ("hbm", 3 * w.H * w.W * n_img + 3 * PH * PW * es * n_planes)
    # descriptors written once, conv5 maps read once
    work["region_windows"] = ("hbm", n_boxes * 256 * 36 * 4 + n_planes * sd[4] ** 2 * 256 * es)
    kind, units = work[dominant]
    launches, tot_ms = live[dominant]
    avg_s = tot_ms / launches / 1e3
    digest = source_digest()
    if kind == "mfma":
        achieved = units / avg_s / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_TFLOPS[dtn],
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_TFLOPS[dtn], 4)}
    else:
        achieved = units / avg_s / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(achieved / PEAK_HBM_GBS, 4)}
    roof["kernel"] = dominant
    roof["avg_launch_ms"] = round(avg_s * 1e3, 4)
    roof["algorithmic_per_launch"] = units
    roof["traffic"] = load_traffic(dominant, w.name, digest)

    conv_ms = sum(breakdown[k][1] / breakdown[k][0] for k in CONV_NAMES if k in breakdown)
    conv_flops = sum(fl) * n_planes
    conv_util = conv_flops / (conv_ms / 1e3) / 1e12 / PEAK_TFLOPS[dtn]

    result = {
        "metric": METRIC, "value": round(value, 2), "unit": "pyramids/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": dtn,
        "data": "synthetic (seeded uniform uint8 images, N(0,0.01) weights, log-uniform boxes)",
        "config": {"workload": w.name, "images": n_img, "image": f"{w.H}x{w.W}",
                   "scales": w.n_scales, "steps_per_octave": w.steps_per_octave,
                   "plane": f"{PH}x{PW}", "planes": n_planes, "boxes_per_image": boxes_per_img,
                   "region_window": "6x6x256"},
        "conv_mfma_util": round(conv_util, 4),
        "conv_tflops": round(conv_flops / (conv_ms / 1e3) / 1e12, 2),
        "roofline": roof,
        "source_digest": digest,
    }
    if args.kernels:
        result["kernels_ms"] = {k: round(v[1] / v[0], 4) for k, v in breakdown.items()}

    if not args.no_per_window:
        result["per_window"] = per_window(D, w, dt, imgs[:1], boxes[:boxes_per_img], packed,
                                          ms_per_step / n_img)
    if not args.no_packed and n_img > 1:
        result["cross_image_packing"] = cross_image(D, w, dt, imgs, boxes, box_img, packed, args.steps,
                                                    args.warmup, ms_per_step)
    if not args.no_single and n_img > 1:
        result["single_image"] = single_image(D, weights, args.steps, args.warmup)
    if not args.no_per_scale and n_img > 1:
        result["per_scale_planes"] = per_scale_planes(D, weights, args.steps, args.warmup)
    if args.ceilings:
        result["ceilings"] = ceilings(D, weights, PH)
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(w, args.cpu_planes)
    print(json.dumps(result), flush=True)


def per_window(D, w, dt, img, boxes, packed, dense_ms_per_image):
    """The per-window baseline the paper compares the dense pyramid with (Sec. 3.4): the 2000 boxes of
    one image each warped to 227 x 227 and run through conv1..conv5 + pool5 on their own (one launch
    per layer over all windows), timed after the main measurement; against the dense path's time per
    image (pyramid, conv stack and 2000 region windows) from the timed steps."""
    import torch

    from paper_1404_1869_amd import workmodel

    n = boxes.shape[0]
    pw = D.PerWindow(n, dt, 227, device=boxes.device)
    for _ in range(2):
        pw(img, boxes, packed, w.mean)
    torch.cuda.synchronize()
    D.profile_start()
    pw(img, boxes, packed, w.mean)
    torch.cuda.synchronize()
    kern = D.profile_stop()
    reps = 5
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        pw(img, boxes, packed, w.mean)
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / reps
    conv_ms = sum(kern[k][1] / kern[k][0] for k in CONV_NAMES if k in kern)
    flops = n * sum(workmodel.conv_flops(227, 227))
    return {"windows": n, "window": "227x227", "ms_per_image": round(ms, 4),
            "dense_ms_per_image": round(dense_ms_per_image, 4),
            "per_window_over_dense": round(ms / dense_ms_per_image, 2),
            "conv_tflops": round(flops / (conv_ms / 1e3) / 1e12, 2),
            "kernels_ms": {k: round(v[1] / v[0], 4) for k, v in kern.items()},
            "paper_context": "Sec. 3.4, NVIDIA K20: 2000 windows ~10 s vs one 25-scale pyramid ~1 s"}


def cross_image(D, w, dt, imgs, boxes, box_img, packed, steps, warmup, per_image_ms):
    """The same step on the same batch with cross-image packing: the rectangles of all images
    stitched together (fewer, fuller planes), the conv stack over the packed planes and the region
    windows read through the packed layout; timed over the same number of steps."""
    import time

    import torch

    n_img = imgs.shape[0]
    plan = D.BatchPlan(n_img, w.H, w.W, D.params_for(w), device=imgs.device)
    planes = D.densenet_build_batch(imgs, plan, dt)
    cf = D.ConvFeatures(plan.planes, dt, D.net_params(pool5=False), device=imgs.device)
    c5d = list(cf.c5d)
    out = torch.empty((boxes.shape[0], 256 * 36), dtype=torch.float32, device=imgs.device)
    scale = torch.empty(boxes.shape[0], dtype=torch.int32, device=imgs.device)

    def step():
        D.densenet_build_batch(imgs, plan, dt, out=planes)
        cf(planes, packed)
        D.densenet_region_windows_batch(cf.conv5, c5d, dt, plan, boxes, box_img, out=out, scale=scale)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    D.profile_start()
    step()
    torch.cuda.synchronize()
    kern = D.profile_stop()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    ms = 1e3 * (time.perf_counter() - t0) / steps
    return {"planes": plan.n_planes, "ms_per_step": round(ms, 4),
            "pyramids_per_s": round(n_img / (ms / 1e3), 2),
            "speedup_vs_per_image_planes": round(per_image_ms / ms, 4),
            "kernels_ms": {k: round(v[1] / v[0], 4) for k, v in kern.items()}}


def single_image(D, weights, steps, warmup):
    """One 25-scale pyramid of one 768 x 1024 image (6 stitched 1200 x 1200 planes, fp16), the unit the
    paper times (Sec. 3.4): ms per pyramid (build + conv stack) launched eagerly and replayed from a
    captured graph of the same launches, the conv MFMA utilisation from traced passes, and the 2000
    region windows of the image timed on their own."""
    import numpy as np
    import torch

    from paper_1404_1869_amd import configs as C
    from paper_1404_1869_amd import synth, workmodel

    w = C.XGA_25SCALE
    dt = D.DTYPES[w.dtypes[0]]
    dev = torch.device("cuda", 0)
    img = torch.from_numpy(synth.images(w.seeds, w.H, w.W)).to(dev)
    packed = D.densenet_pack_weights(weights, dt)
    params = D.params_for(w)
    planes, plan = D.densenet_build_pyramid(img, params, dt)
    cf = D.ConvFeatures(list(plan.planes), dt, D.net_params(pool5=False), device=dev)
    c5d = list(cf.c5d)
    boxes = torch.from_numpy(synth.boxes(w.box_seed or 105, 2000, w.H, w.W)).to(dev)
    out = torch.empty((2000, 256 * 36), dtype=torch.float32, device=dev)
    scale = torch.empty(2000, dtype=torch.int32, device=dev)
    ppi = len(plan.planes)

    def pyramid():
        D.densenet_build_pyramid(img, params, dt, out=planes)
        cf(planes, packed)

    def regions():
        D.densenet_region_windows(cf.conv5, c5d, dt, plan, w.pad, ppi, boxes, out=out, scale=scale)

    def timed(fn, n):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record()
        for _ in range(n):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / n

    for _ in range(warmup):
        pyramid()
        regions()
    torch.cuda.synchronize()
    D.profile_start()  # per-kernel times averaged over `steps` traced pyramids
    for _ in range(steps):
        pyramid()
    torch.cuda.synchronize()
    kern = D.profile_stop()
    eager_ms = timed(pyramid, steps)
    regions_ms = timed(regions, steps)

    # the same launches captured once into a graph (no allocation or memset inside), replayed
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        pyramid()
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        pyramid()
    for _ in range(warmup):
        graph.replay()
    graph_ms = timed(graph.replay, steps)

    fl = workmodel.conv_flops(plan.planes[0].h, plan.planes[0].w)
    conv_ms = sum(kern[k][1] / kern[k][0] for k in CONV_NAMES if k in kern)
    conv_flops = sum(fl) * ppi
    best = min(eager_ms, graph_ms)
    return {"workload": w.name, "dtype": w.dtypes[0], "planes": ppi,
            "ms_per_pyramid_eager": round(eager_ms, 4), "ms_per_pyramid_graph": round(graph_ms, 4),
            "pyramids_per_s": round(1e3 / best, 2),
            "conv_mfma_util": round(conv_flops / (conv_ms / 1e3) / 1e12 / PEAK_TFLOPS[w.dtypes[0]], 4),
            "regions_2000_ms": round(regions_ms, 4),
            "kernels_ms": {k: round(v[1] / v[0], 4) for k, v in kern.items()},
            "paper_context": "Sec. 3.4, NVIDIA K20: one 25-scale pyramid in ~1 s"}


def per_scale_planes(D, weights, steps, warmup):
    """The workloads that give each scale its own plane (Sec. 3.1 without stitching): a 480 x 640 image
    at 8 scales (8 plane sizes; fp16 and fp32) and a 227 x 227 image at 2 scales with pool5 (fp32).
    Per workload: ms per pyramid (build + conv stack, eager, inputs resident), pyramids/s, and the conv
    MFMA utilisation against the dtype's peak (algorithmic conv work of every plane over the summed
    conv kernel time of traced pyramids).  Every layer is one launch over all plane sizes."""
    import torch

    from paper_1404_1869_amd import configs as C
    from paper_1404_1869_amd import synth, workmodel

    dev = torch.device("cuda", 0)
    out = {}
    for w in (C.VGA_8SCALE, C.ALEXNET_227):
        img = torch.from_numpy(synth.images(w.seeds, w.H, w.W)).to(dev)
        params = D.params_for(w)
        res = {}
        for dtn in w.dtypes:
            dt = D.DTYPES[dtn]
            packed = D.densenet_pack_weights(weights, dt)
            planes, plan = D.densenet_build_pyramid(img, params, dt)
            cf = D.ConvFeatures(list(plan.planes), dt, D.net_params(pool5=w.pool5), device=dev)

            def pyramid():
                D.densenet_build_pyramid(img, params, dt, out=planes)
                cf(planes, packed)

            for _ in range(warmup):
                pyramid()
            torch.cuda.synchronize()
            D.profile_start()
            for _ in range(steps):
                pyramid()
            torch.cuda.synchronize()
            kern = D.profile_stop()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            for _ in range(steps):
                pyramid()
            b.record()
            torch.cuda.synchronize()
            ms = a.elapsed_time(b) / steps
            conv_ms = sum(kern[k][1] for k in CONV_NAMES if k in kern) / steps
            flops = sum(sum(workmodel.conv_flops(d.h, d.w)) for d in plan.planes)
            res[dtn] = {"planes": [f"{d.h}x{d.w}" for d in plan.planes], "ms_per_pyramid": round(ms, 4),
                        "pyramids_per_s": round(1e3 / ms, 2),
                        "conv_launches_per_pyramid": round(sum(kern[k][0] for k in CONV_NAMES if k in kern)
                                                           / steps, 2),
                        "conv_mfma_util": round(flops / (conv_ms / 1e3) / 1e12 / PEAK_TFLOPS[dtn], 4)}
        out[w.name] = res
    return out


def mfma_chain(timed):
    """Sustained rate of independent v_mfma_f32_32x32x16_bf16 chains with no memory traffic
    (libprobe.so), two waves per SIMD on every SIMD: every MFMA reading the same registers of smooth
    values (the most favourable case), random bit patterns in four register sets read in turn, and
    the smooth values copied into four register sets read in turn.  The matrix cores' ceiling on
    this device and how far it moves with the operands."""
    import ctypes

    import torch

    path = os.path.join(ROOT, "paper_1404_1869_amd", "libprobe.so")
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: run __graft_entry__.build() first")
    lib = ctypes.CDLL(path)
    fn = lib.densenet_probe_mfma_bf16
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_int64,
                   ctypes.POINTER(ctypes.c_double), ctypes.c_void_p]
    n_out = 2 * torch.cuda.get_device_properties(0).multi_processor_count * 256
    buf = torch.empty(n_out, dtype=torch.float32, device="cuda")
    flop = ctypes.c_double()
    res = {}
    for mode, name in ((0, "repeated_registers_smooth_values"), (1, "random"),
                       (2, "rotated_registers_smooth_values")):
        def launch(k):
            st = fn(mode, k, buf.data_ptr(), n_out, ctypes.byref(flop),
                    ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
            if st != 0:
                raise RuntimeError("MFMA probe launch failed")
        launches = 100
        s = timed(lambda: launch(launches), 1, 1)
        res[name] = round(flop.value * launches / s / 1e12, 1)
    del buf
    return res


def ceilings(D, weights, plane_side):
    """Device ceilings under the same conditions as the kernels (context for the roofline figures).

    * mfma_chain_bf16_tflops: chains of dense bf16 MFMAs with no memory traffic (see mfma_chain).
    * gemm_bf16_tflops: torch.mm of two 8192 x 8192 bf16 matrices (the vendor GEMM library), on
      N(0, 1) operands and on zeros.  The matrix cores' sustained rate depends on the operand values
      (the clock falls under the power drawn by toggling data), so the zero-operand figure is the
      nearest to the 2.5 PF datasheet peak and the random one to what real data allows.
    * conv_96_planes: this library's conv2 and conv3 over 96 planes of the default workload's map
      sizes, on N(0, 10)-magnitude inputs with the N(0, 0.01) weights and on zero inputs and weights;
      conv1 over 96 planes of uniform +-128 values with those weights and with zero weights.
    * hbm_tbs: a 1 GiB device-to-device copy (read + write) and a 1 GiB fill.
    """
    import numpy as np
    import torch

    from paper_1404_1869_amd import workmodel

    def timed(fn, reps, warm):
        for _ in range(warm):
            fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        b.synchronize()
        return a.elapsed_time(b) / reps / 1e3  # seconds

    out = {}
    g = torch.Generator(device="cuda").manual_seed(11)
    n = 8192
    gemm = {}
    for name, make in (("random", lambda: torch.randn((n, n), device="cuda", generator=g)),
                       ("zero", lambda: torch.zeros((n, n), device="cuda"))):
        a = make().to(torch.bfloat16).contiguous()
        b = make().to(torch.bfloat16).contiguous()
        c = torch.empty((n, n), device="cuda", dtype=torch.bfloat16)
        s = timed(lambda: torch.mm(a, b, out=c), 30, 10)
        gemm[name] = round(2.0 * n ** 3 / s / 1e12, 1)
        del a, b, c
    out["gemm_bf16_tflops"] = gemm
    out["mfma_chain_bf16_tflops"] = mfma_chain(timed)

    bf = D.DTYPES["bf16"]
    zero_w = [(torch.zeros_like(wt), bs) for wt, bs in weights]
    packs = {"real": D.densenet_pack_weights(weights, bf), "zero": D.densenet_pack_weights(zero_w, bf)}
    sd = workmodel.sides(plane_side)
    fl = workmodel.conv_flops(plane_side, plane_side)
    conv = {}
    for layer, C, H in ((2, 96, sd[1]), (3, 256, sd[3])):
        shp = (96, H, H, C)
        xs = {"random": (torch.randn(shp, device="cuda", generator=g) * 10).abs().to(torch.bfloat16),
              "zero": torch.zeros(shp, device="cuda", dtype=torch.bfloat16)}
        for name in ("random", "zero"):
            x, p = xs[name], packs["real" if name == "random" else "zero"]
            s = timed(lambda: D.densenet_conv_layer(layer, x, 96, H, H, bf, p), 10, 3)
            conv[f"conv{layer}_{name}_us"] = round(s * 1e6, 1)
            conv[f"conv{layer}_{name}_tflops"] = round(fl[layer - 1] * 96 / s / 1e12, 1)
        del xs
    # conv1 over 96 planes of 1200 x 1200 (channel-major, rows a multiple of 8: the direct-load
    # kernel): uniform +-128 planes with the N(0, 0.01) weights, and the same planes with zero weights
    xp = ((torch.rand((96, 3, plane_side, plane_side), device="cuda", generator=g) - 0.5) * 256).to(torch.bfloat16)
    for name in ("random", "zero_weights"):
        p = packs["real" if name == "random" else "zero"]
        s = timed(lambda: D.densenet_conv_layer(1, xp, 96, plane_side, plane_side, bf, p), 10, 3)
        conv[f"conv1_{name}_us"] = round(s * 1e6, 1)
        conv[f"conv1_{name}_tflops"] = round(fl[0] * 96 / s / 1e12, 1)
    del xp
    out["conv_96_planes"] = conv
    torch.cuda.empty_cache()

    nb = 1 << 30
    src = torch.empty(nb, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    src.fill_(1)
    out["hbm_tbs"] = {"copy": round(2.0 * nb / timed(lambda: dst.copy_(src), 10, 3) / 1e12, 2),
                      "fill": round(nb / timed(lambda: dst.fill_(2), 10, 3) / 1e12, 2)}
    del src, dst
    torch.cuda.empty_cache()
    return out


def cpu_model() -> str:
    """The host CPU as /proc/cpuinfo names it (model name, family / model / stepping of the first
    processor entry) and the logical CPUs this process may run on."""
    fields = {}
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if not line.strip():
                    break  # first processor entry only
                if ":" in line:
                    k, v = line.split(":", 1)
                    fields.setdefault(k.strip(), v.strip())
    except OSError:
        pass
    name = fields.get("model name", "unknown")
    fam = [f"{k} {fields[k]}" for k in ("cpu family", "model", "stepping") if k in fields]
    try:
        usable = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        usable = os.cpu_count() or 0
    return f"{name} ({', '.join(fam)}; {usable} logical CPUs usable)" if fam else f"{name} ({usable} logical CPUs usable)"


def cpu_baseline(w, n_planes_sample):
    """The oracle, as it stands, on a bounded sample of the workload: image 0's planes and its 2000
    region windows in full, its conv stack on `n_planes_sample` of its planes (a plane's cost depends
    only on its size), extrapolated to one 25-scale pyramid."""
    import numpy as np

    import oracle
    from paper_1404_1869_amd import synth

    img = synth.image(w.seeds[0], w.H, w.W)
    W7 = synth.weights(7)
    t0 = time.perf_counter()
    p = oracle.plan(w.H, w.W, w.n_scales, w.steps_per_octave, w.base_scale, w.base_longest_side,
                    w.pad, w.plane_h, w.plane_w)
    planes = oracle.build_planes(img, p, w.pad_mode, w.mean)
    t_build = time.perf_counter() - t0
    c5 = {}
    t0 = time.perf_counter()
    for j in range(n_planes_sample):
        c5[j] = oracle.net(planes[j].astype(np.float32), W7)
    t_plane = (time.perf_counter() - t0) / n_planes_sample
    maps = [c5.get(j, np.zeros((256, oracle.conv5_side(h), oracle.conv5_side(wd)), np.float32))
            for j, (h, wd) in enumerate(p.plane_sizes)]
    boxes = synth.boxes(105, 2000, w.H, w.W)
    t0 = time.perf_counter()
    oracle.region_windows(maps, p, boxes)
    t_reg = time.perf_counter() - t0
    per_pyr = t_build + p.n_planes * t_plane + t_reg
    return {"value": round(1.0 / per_pyr, 5), "unit": "pyramids/s", "cores": oracle.threads(),
            "cpu": cpu_model(), "kind": "oracle",
            "sample": (f"image 0 of the workload: planes and 2000 region windows in full, conv stack "
                       f"on {n_planes_sample} of its {p.n_planes} 1200x1200 planes, extrapolated to "
                       f"{p.n_planes} planes ({per_pyr:.1f} s per pyramid)")}


if __name__ == "__main__":
    main()

"""Benchmark: integer TOPS and ms/image of the fully-quantized RetinaNet-R50
(ResNet-50 without the stem + FPN + RetinaNet heads, 4-bit codes, batch 8,
800 x 1333 images) on one MI355X, through the C ABI.

One step = one forward pass of all 110 convolution segments over the batch
(grouped launches on one HIP stream, recorded once into a HIP graph and
replayed), inputs resident in HBM; each replay is bracketed by HIP events
(mean, median, p10 and p90 per step). The dominant kernel is the grouped
head-tower launch (3x3, 256 -> 256, class and box towers, five pyramid
levels, eight images); a second timed pass enqueues the same steps launch by
launch on one stream, with HIP events on that stream around every grouped
launch: the per-launch table (integer TOPS, GB/s against algorithmic bytes,
fraction of the binding MFMA or HBM roof) and the head-tower launch time of
the roofline. Each head-tower launch is also repeated back to back between
two events (`back_to_back_us`): sustained, with no lighter launch between,
the same kernel runs a few percent slower (the clock drops under the load).

Prints one JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "int TOPS per qconv layer + ms/image quantized RetinaNet-R50 800x1333, 1 GPU"
MFMA_I8_PEAK_TOPS = 5000.0  # MI355X dense int8 MFMA
MFMA_FP4_PEAK_TOPS = 10100.0  # MI355X dense FP4 MFMA
HBM_PEAK_GBS = 8000.0       # MI355X HBM3E
COPY_PROBE_BYTES = 256 << 20
B2B_REPS = 10               # back-to-back repeats of each dominant launch (sustained load)

# HBM traffic of one head-tower launch, from two rocprofv3 counter runs
# (FETCH_SIZE, WRITE_SIZE) scaled by the same counters on a plain copy of
# COPY_PROBE_BYTES; valid only for the kernel source it was measured on.
HEAD_KERNEL = "qconv_wv_kernel<0, 0, 1, 8>"
HEAD_KERNEL_SOURCES = ("qconv_wv.hip", "mfma_common.h")
HEAD_TRAFFIC = {"kernel_sha256": "402e1eba8ec83cff12c1afac0d594bd7148c0230c8e3c31c2a82a2e48be5d333",
                "fetch_bytes": 51036641, "write_bytes": 45670400}


def kernel_sha256():
    """Hash of the dominant kernel's sources (the kernel and its helpers)."""
    import hashlib
    h = hashlib.sha256()
    for name in HEAD_KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2007_06919_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_peaks(torch, dev):
    """The ceilings measured on this GPU next to the published figures: the
    int8 matrix-core rate of a kernel of MFMAs alone (aqd_mfma_probe: two
    workgroups of 4 waves per CU, operands of 4-bit magnitudes) and the HBM
    rate of a device-to-device copy of COPY_PROBE_BYTES (read + write)."""
    from paper_2007_06919_amd import aqd
    wgs, iters = 2048, 1000
    out = torch.empty(wgs * 256, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream()
    aqd.mfma_probe(wgs, iters, out, stream)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(5):
        aqd.mfma_probe(wgs, iters, out, stream)
    e1.record(stream)
    torch.cuda.synchronize()
    mfma_ms = e0.elapsed_time(e1) / 5
    mfma_tops = wgs * 4 * iters * 16 * 32768 / (mfma_ms / 1e3) / 1e12
    src = torch.ones(COPY_PROBE_BYTES, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    e0.record(stream)
    for _ in range(5):
        dst.copy_(src)
    e1.record(stream)
    torch.cuda.synchronize()
    copy_ms = e0.elapsed_time(e1) / 5
    del src, dst, out
    log(f"[bench] measured ceilings: int8 MFMA {mfma_tops:.0f} TOPS, HBM copy "
        f"{2 * COPY_PROBE_BYTES / (copy_ms / 1e3) / 1e9:.0f} GB/s")
    return {"mfma_i8_tops": round(mfma_tops, 1),
            "hbm_copy_gbs": round(2 * COPY_PROBE_BYTES / (copy_ms / 1e3) / 1e9, 1),
            "mfma_probe": f"aqd_mfma_probe, {wgs} workgroups x 4 waves x {iters} x 16 MFMAs 16x16x64 i8, "
                          f"mean of 5 launches",
            "hbm_probe": f"device copy of {COPY_PROBE_BYTES} bytes (read + write), mean of 5"}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def cpu_baseline(bits=4):
    """The oracle on a bounded sample of every workload: one image of each
    (the calibration image; both images of the literal basic block), the
    whole network per image, seeded inputs and parameters as on the GPU.
    value: the oracle's integer-op rate on the sample of the timed workload
    (one of its eight images); per_config: the oracle's wall time per sample
    and the time the whole workload would take at that rate."""
    from oracle import network, ref
    from paper_2007_06919_amd import workloads

    per, main = {}, None
    for idx, name in enumerate(workloads.CONFIG_NAMES):
        if bits != 4 and idx == 4:
            net, params = workloads.retinanet_config(8, 800, 1333, bits)
            name = f"retinanet_r50_fpn_n8_800x1333_{bits}bit"
        else:
            net, params = workloads.config(idx)
        n = net.tensors[net.inputs[0]].n
        images = list(range(n)) if params.mode == "literal" else sorted(set(params.calib_images))
        t0 = time.perf_counter()
        network.run(net, params, images=images, keep=set())
        wall = time.perf_counter() - t0
        macs = net.total_macs() * len(images) // n
        per[name] = {"images": f"{len(images)} of {n}", "wall_s": round(wall, 3),
                     "full_wall_s": round(wall * n / len(images), 3),
                     "int_tops": round(2 * macs / wall / 1e12, 5)}
        log(f"[bench] oracle {name}: {len(images)} of {n} images in {wall:.2f} s")
        if idx == 4:
            main = (2 * macs / wall / 1e12, name, len(images), n, wall)
    tops, name, k, n, wall = main
    return {"value": round(tops, 5), "unit": "int TOPS", "cores": ref.num_threads(),
            "kind": "oracle",
            "sample": f"{name}: {k} of {n} images through the whole network ({wall:.1f} s); "
                      f"the other workloads one image each (per_config)",
            "per_config": per}


def launch_cost(gpu, group):
    """(integer ops, algorithmic HBM bytes) of one grouped launch: every input
    code, weight, skip operand and output read or written once. A fused
    projection shortcut adds its own input and weights; its int32 output is
    never materialised."""
    from paper_2007_06919_amd import aqd
    net = gpu.net
    sb = aqd.stored_bits

    def tbytes(name):
        t = net.tensors[name]
        return t.n * t.h * t.w * t.c * (32 if t.bits == 32 else sb(t.bits)) // 8

    macs, nbytes, seen = 0, 0, set()
    for conv, si in group:
        x, skip, y = conv.segs[si]
        if conv.op != "conv":
            nbytes += tbytes(x) + tbytes(y)
            continue
        ty = net.tensors[y]
        macs += ty.n * ty.h * ty.w * conv.cout * conv.k * conv.k * conv.cin
        nbytes += tbytes(x) + tbytes(y)
        if conv.name not in seen:
            nbytes += conv.k * conv.k * conv.cin * conv.cout * sb(conv.bits_w) // 8
            seen.add(conv.name)
        proj = gpu.fused.get(conv.name)
        if proj is not None:
            px, _, py = proj.segs[0]
            tp = net.tensors[py]
            macs += tp.n * tp.h * tp.w * proj.cout * proj.cin
            nbytes += tbytes(px) + proj.cin * proj.cout * sb(proj.bits_w) // 8
        elif skip is not None:
            nbytes += tbytes(skip)
    return 2 * macs, nbytes


def pct(v, q):
    import numpy as np
    return float(np.percentile(np.asarray(v), q))


def fp4_layer(args):
    """The 2-bit head-tower launch (class and box towers' 3x3 256 -> 256 layer
    over P3-P7 of a batch of eight 800x1333 images: 10 segments, one grouped
    launch) on the FP4 MFMA path and on the int8 MFMA path (handles created
    with AQD_NO_FP4=1); both outputs must agree byte for byte."""
    import numpy as np
    import torch
    from paper_2007_06919_amd import aqd, workloads

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.Stream(device=dev)
    sizes = workloads.pyramid_sizes(800, 1333)
    n = 8
    rng = np.random.Generator(np.random.PCG64(2))
    cases = [workloads.random_conv_case(seed=70 + t, n=1, h=8, w=8, cin=256, cout=256, k=3, bits_in=2,
                                        bits_w=2, wenc=workloads.WENC_PAPER_ODD, bits_out=2,
                                        num_levels=len(sizes)) for t in range(2)]
    xs = [torch.from_numpy(aqd.pack_codes(rng.integers(0, 4, size=(n, h, w, 256)), 2)).to(dev)
          for h, w in sizes]

    def handles(no_fp4):
        old = os.environ.get("AQD_NO_FP4")
        os.environ["AQD_NO_FP4"] = "1" if no_fp4 else "0"
        try:
            return [aqd.qconv_create(256, 256, 3, 1, 1, 2, 2, aqd.pack_codes(c.w_fields, 2), c.levels,
                                     wenc=workloads.WENC_PAPER_ODD, bits_out=2) for c in cases]
        finally:
            if old is None:
                del os.environ["AQD_NO_FP4"]
            else:
                os.environ["AQD_NO_FP4"] = old

    out, res = {}, {}
    for name, no_fp4 in (("fp4", False), ("int8", True)):
        hs = handles(no_fp4)
        try:
            paths = {aqd.qconv_path(h) for h in hs}
            ys = [[torch.empty((n, h, w, 64), dtype=torch.uint8, device=dev) for h, w in sizes]
                  for _ in hs]
            segs = [(hs[t], lv, n, h, w, xs[lv], None, 0, 0, ys[t][lv])
                    for t in range(2) for lv, (h, w) in enumerate(sizes)]
            with torch.cuda.stream(stream):
                for _ in range(args.warmup):
                    aqd.qconv_run_group(segs, stream)
                stream.synchronize()
                ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                      for _ in range(args.steps)]
                for e0, e1 in ev:
                    e0.record(stream)
                    aqd.qconv_run_group(segs, stream)
                    e1.record(stream)
                stream.synchronize()
            us = [1e3 * e0.elapsed_time(e1) for e0, e1 in ev]
            res[name] = {"path": sorted(paths), "us_median": round(float(np.median(us)), 2),
                         "us_p10": round(pct(us, 10), 2), "us_p90": round(pct(us, 90), 2)}
            out[name] = [y.cpu().numpy() for row in ys for y in row]
            log(f"[bench] {name}: {res[name]}")
        finally:
            for h in hs:
                aqd.qconv_destroy(h)
    assert all(np.array_equal(a, b) for a, b in zip(out["fp4"], out["int8"])), "FP4 and int8 paths differ"
    ops = 2 * 2 * sum(n * h * w for h, w in sizes) * 256 * 9 * 256
    for name, peak in (("fp4", MFMA_FP4_PEAK_TOPS), ("int8", MFMA_I8_PEAK_TOPS)):
        tops = ops / (res[name]["us_median"] * 1e-6) / 1e12
        res[name].update(int_tops=round(tops, 1), peak_tops=peak, frac=round(tops / peak, 4))
    print(json.dumps({"metric": "2-bit head-tower launch: FP4 MFMA path vs int8 MFMA path",
                      "unit": "us", "steps": args.steps, "warmup": args.warmup, "int_ops_per_launch": ops,
                      "config": {"workload": "retina_head_towers_p3p7_n8_800x1333_2bit", "batch": n,
                                 "segments": 10},
                      "outputs_equal": True, "speedup": round(res["int8"]["us_median"] / res["fp4"]["us_median"], 3),
                      **res}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--bits", type=int, default=4, choices=(3, 4),
                    help="code width of the network (3: the paper's 3-bit RetinaNet, codes in "
                         "4-bit containers; the default 4 is the benchmarked workload)")
    ap.add_argument("--io-bits", type=int, default=0, choices=(0, 8),
                    help="8: the fully quantized network of the paper's AQD rows (Sec. 4): 8-bit image, "
                         "7x7 stem and prediction convolutions, max-pooling; 0: the network from the "
                         "max-pooled stem output on, predictions at the network's width")
    ap.add_argument("--fp4-layer", action="store_true",
                    help="instead of the network: the 2-bit head-tower launch (3x3 256->256, class "
                         "and box towers, P3-P7, batch 8, 800x1333) on the FP4 MFMA path and on the "
                         "int8 MFMA path, timed launch by launch")
    ap.add_argument("--copy-probe", action="store_true",
                    help="after the run, one device copy of 256 MiB (a kernel of known traffic "
                         "for calibrating memory counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); several GPUs "
              f"would each take whole images of the batch, which is not run here.", file=sys.stderr)
        sys.exit(2)
    import faulthandler
    faulthandler.enable()      # a crash prints the Python stack of every thread
    if args.fp4_layer:
        fp4_layer(args)
        return

    import numpy as np
    import torch
    from paper_2007_06919_amd import runner, workloads

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    t0 = time.time()
    if args.io_bits:
        net, params = workloads.retinanet_config(8, 800, 1333, args.bits, io_bits=args.io_bits)
        workload = f"retinanet_r50_fpn_n8_800x1333_{args.bits}bit_io{args.io_bits}"
    elif args.bits == 4:
        net, params = workloads.config(4)
        workload = workloads.CONFIG_NAMES[4]
    else:
        net, params = workloads.retinanet_config(8, 800, 1333, args.bits)
        workload = f"retinanet_r50_fpn_n8_800x1333_{args.bits}bit"
    log(f"[bench] workload drawn in {time.time() - t0:.1f} s; "
        f"{len(net.convs)} convs, {sum(len(c.segs) for c in net.convs)} segments")
    t0 = time.time()
    stream = torch.cuda.Stream(device=dev)
    with torch.cuda.stream(stream):
        gpu = runner.Net(net, params, device="cuda:0", stream=stream)
    log(f"[bench] handles created and calibrated in {time.time() - t0:.1f} s; "
        f"{gpu.launches_per_forward()} launches per step, {len(gpu.fused)} projection shortcuts fused")

    n_img = net.tensors[net.inputs[0]].n
    total_ops = 2 * net.total_macs()
    live = [gi for gi in range(len(gpu.schedule)) if gpu.lane[gi] is not None]
    cost = {gi: launch_cost(gpu, gpu.schedule[gi]) for gi in live}
    dominant = [gi for gi in live if gpu.schedule[gi][0][0].k == 3
                and gpu.schedule[gi][0][0].cin == 256 and gpu.schedule[gi][0][0].cout == 256
                and gpu.schedule[gi][0][0].name.startswith(("cls.t", "box.t"))]
    from paper_2007_06919_amd import aqd
    path = {gi: aqd.qconv_path(gpu.handles[gpu.schedule[gi][0][0].name])
            if gpu.schedule[gi][0][0].op == "conv" else gpu.schedule[gi][0][0].op for gi in live}
    peak = {gi: MFMA_FP4_PEAK_TOPS if path[gi] == "fp4-mfma" else MFMA_I8_PEAK_TOPS for gi in live}
    events = {}

    def hook(gi, when, s):
        ev = torch.cuda.Event(enable_timing=True)
        ev.record(s)
        events.setdefault(gi, []).append(ev)

    with torch.cuda.stream(stream):
        for _ in range(args.warmup):
            gpu.forward(stream)
        stream.synchronize()
        log(f"[bench] {args.warmup} eager warm-up passes done")
        # the whole network recorded once into a HIP graph; a step = one replay
        gpu.capture(stream)
        for _ in range(args.warmup):
            gpu.replay()
        stream.synchronize()
        torch.cuda.synchronize()
        log(f"[bench] graph captured, {args.warmup} warm-up replays done")
        marks = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
        wall0 = time.perf_counter()
        marks[0].record(stream)
        for i in range(args.steps):
            gpu.replay()
            marks[i + 1].record(stream)
        stream.synchronize()
        torch.cuda.synchronize()
        wall = time.perf_counter() - wall0
        log(f"[bench] {args.steps} timed replays done")
        # the dominant launches again, each B2B_REPS times back to back between
        # two events on the launch stream (sustained load); before the
        # launch-by-launch pass, so that a kernel trace ends with that pass
        b0 = torch.cuda.Event(enable_timing=True)
        b1 = torch.cuda.Event(enable_timing=True)
        b0.record(stream)
        for gi in dominant:
            for _ in range(B2B_REPS):
                gpu.launch_group(gi, stream)
        b1.record(stream)
        stream.synchronize()
        torch.cuda.synchronize()
        # the same steps launch by launch on one stream (no overlap), with
        # events on the launch stream around every grouped launch
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(args.steps):
            gpu.forward(stream, launch_hook=hook, serial=True)
        e1.record(stream)
        stream.synchronize()
        torch.cuda.synchronize()
    step_ms = [marks[i].elapsed_time(marks[i + 1]) for i in range(args.steps)]
    ms_step = marks[0].elapsed_time(marks[-1]) / args.steps
    serial_ms_step = e0.elapsed_time(e1) / args.steps
    value = total_ops / (ms_step / 1e3) / 1e12

    launch_us = {gi: [1e3 * evs[k].elapsed_time(evs[k + 1]) for k in range(0, len(evs), 2)]
                 for gi, evs in events.items()}
    per_launch = []
    for gi in live:
        ops, nbytes = cost[gi]
        us = float(np.median(launch_us[gi]))
        t_mfma = ops / (peak[gi] * 1e12) * 1e6
        t_hbm = nbytes / (HBM_PEAK_GBS * 1e9) * 1e6
        bound = "mfma" if t_mfma >= t_hbm else "hbm"
        conv0 = gpu.schedule[gi][0][0]
        per_launch.append({
            "launch": "+".join(sorted({c.name for c, _ in gpu.schedule[gi]})),
            "segments": len(gpu.schedule[gi]), "shape": f"{conv0.k}x{conv0.k} {conv0.cin}->{conv0.cout}",
            "path": path[gi],
            "us": round(us, 2), "int_tops": round(ops / us / 1e6, 1),
            "gbs": round(nbytes / us / 1e3, 1), "bound": bound,
            "frac": round(max(t_mfma, t_hbm) / us, 4),
            "mfma_frac": round(t_mfma / us, 4), "hbm_frac": round(t_hbm / us, 4)})

    durs = [u for gi in dominant for u in launch_us[gi]]
    avg_ops = float(np.mean([cost[gi][0] for gi in dominant]))
    avg_us = float(np.mean(durs))
    b2b_us = 1e3 * b0.elapsed_time(b1) / (B2B_REPS * len(dominant))
    achieved = avg_ops / (avg_us / 1e6) / 1e12
    dom_peak = peak[dominant[0]]
    log(f"[bench] {ms_step:.3f} ms/step as a graph replay (median {np.median(step_ms):.3f}, "
        f"p10 {pct(step_ms, 10):.3f}, p90 {pct(step_ms, 90):.3f}; wall "
        f"{wall / args.steps * 1e3:.3f} ms; {serial_ms_step:.3f} ms launch by launch on one "
        f"stream), {value:.1f} int TOPS; head-tower launch {avg_us:.1f} us, {achieved:.1f} TOPS")

    out = {
        "metric": METRIC, "value": round(value, 3), "unit": "int TOPS", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "i8", "data": "synthetic",
        "config": {"workload": workload, "batch": n_img, "image": [800, 1333],
                   "bits": args.bits, "conv_segments": sum(len(c.segs) for c in net.convs),
                   "launches_per_step": gpu.launches_per_forward(), "int_ops_per_step": total_ops,
                   "hip_graph": True},
        "ms_per_image": round(ms_step / n_img, 4),
        "step_ms": {"mean": round(ms_step, 4), "median": round(float(np.median(step_ms)), 4),
                    "p10": round(pct(step_ms, 10), 4), "p90": round(pct(step_ms, 90), 4),
                    "replays": args.steps},
        "serial_ms_per_step": round(serial_ms_step, 4),
        "roofline": {"bound": "mfma",
                     "kernel": f"{HEAD_KERNEL} (head towers 3x3 256->256, 10 segments, "
                               f"256x128 tiles)",
                     "achieved": round(achieved, 2), "peak": dom_peak, "unit": "TOPS",
                     "frac": round(achieved / dom_peak, 4), "traffic": None,
                     "avg_launch_us": round(avg_us, 2), "ops_per_launch": int(avg_ops),
                     "launch_us_p10_p50_p90": [round(pct(durs, q), 2) for q in (10, 50, 90)],
                     "timing": "HIP events on the launch stream around each head-tower launch of the "
                               "launch-by-launch pass (the dispatch gap included)",
                     "back_to_back_us": round(b2b_us, 2)},
        "per_launch": per_launch,
    }
    traffic = None
    if args.bits == 4 and HEAD_TRAFFIC and HEAD_TRAFFIC["kernel_sha256"] == kernel_sha256():
        traffic = HEAD_TRAFFIC["fetch_bytes"] + HEAD_TRAFFIC["write_bytes"]
    out["roofline"]["traffic"] = traffic
    gpu.close()
    out["measured_peaks"] = measured_peaks(torch, dev)
    out["roofline"]["frac_of_measured_mfma"] = round(achieved / out["measured_peaks"]["mfma_i8_tops"], 4)
    if args.copy_probe:
        src = torch.ones(COPY_PROBE_BYTES, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] copy probe: {COPY_PROBE_BYTES} bytes device to device")
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a bounded sample ...")
        out["cpu_baseline"] = cpu_baseline(args.bits)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

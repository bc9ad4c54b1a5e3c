"""Benchmark of block-swapped inference on one MI355X.

One step = one inference of the whole hot path over one input: every slab
streamed from the pinned host image into the budgeted HBM arena (one DMA per
slab, copy stream), bound by pointer, computed by the HIP kernels on the
compute stream, its range reused by the slab two places later.  The network
input is resident in HBM when the timed region starts; the weights are in
pinned host memory, as the method intends.

Prints ONE JSON line with
  value     swapped / all-resident latency ratio (lower is better);
  h2d_*     streamed weight bytes per second vs the measured pinned-H2D peak;
  roofline  the dominant compute kernel against the MFMA fp16 peak;
  link      the swap DMA against the measured pinned-H2D peak;
  cpu_baseline  the fp64 CPU oracle on this host (a baseline, not a target).

Usage: python bench.py [--gpus 1] [--steps 20] [--warmup 3] [--workload resnet50]
"""
import argparse
import gc
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

MFMA_FP16_PEAK_TFLOPS = 2500.0     # MI355X dense fp16 MFMA
PMC_INFERENCES = 5                 # resident inferences between the counter markers
HBM_PEAK_GBS = 8000.0
METRIC = "swapped/all-resident latency ratio at budget; H2D GB/s vs link peak; MFMA util"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="resnet50",
                    choices=["tiny_cnn", "resnet50", "vgg16", "fcn_resnet101", "decoder7b"])
    ap.add_argument("--gen-tokens", type=int, default=None,
                    help="decoder: tokens generated after the prompt (default 128)")
    ap.add_argument("--budget-frac", type=float, default=None,
                    help="budget as a fraction of the weight bytes (default: the workload's)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="approximate CPU time spent on the oracle baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--verbose", action="store_true")
    ap.add_argument("--no-graph", action="store_true", help="enqueue call by call (no HIP graph)")
    ap.add_argument("--swapin", type=int, default=2, choices=[0, 1, 2],
                    help="0 copy kernel, 1 SDMA from the calling thread, 2 SDMA from the copy thread")
    ap.add_argument("--partition", type=int, default=3, choices=[0, 1, 2, 3],
                    help="0: slabs follow the workload's blocks; 1: balanced re-cut into "
                         "ceil(2 s / B) equal slabs; 2: searched under a delay model "
                         "calibrated on this GPU (on the workload-block plan, untimed); "
                         "3 (default): the fastest of 0, 1, 2 measured on this GPU "
                         "(sn_tune, untimed)")
    ap.add_argument("--sync", type=int, default=2, choices=[0, 1, 2],
                    help="copy thread ordering: 0 events + signal kernels, "
                         "1 stream write/wait of values in mapped memory, "
                         "2 ROCr SDMA copies with a gate kernel polling each slab's completion signal")
    ap.add_argument("--copy-streams", type=int, default=1, choices=[1, 2],
                    help="DMA queues used by the copy thread (consecutive slabs alternate)")
    ap.add_argument("--swapin-blocks", type=int, default=None,
                    help="workgroups of the copy kernel (--swapin 0)")
    ap.add_argument("--ablation", action="store_true",
                    help="also time the naive swapping modes (SN_OPT_NAIVE), untimed in `value`")
    ap.add_argument("--image-file", default=None, metavar="PATH",
                    help="storage tier: write the swapped plan's image to PATH, swap in from it "
                         "with direct I/O (sn_attach_image_file) and report the storage read "
                         "rate against the file's raw O_DIRECT read rate")
    ap.add_argument("--link-sweep", action="store_true",
                    help="only measure the pinned host -> device copy rate for sizes 4 KiB .. "
                         "1 GiB (median of 20 each; one JSON line per size)")
    ap.add_argument("--pmc-calibration", action="store_true",
                    help="for counter runs: after the timed work, run a 256 MiB device-to-device "
                         "copy (calibration and start marker), %d all-resident inferences and a "
                         "64 MiB copy (end marker)" % PMC_INFERENCES)
    ap.add_argument("--pmc-summary", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="no GPU: summarise two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE) of "
                         "'bench.py --pmc-calibration' into profiles/<kernel>_<workload>_traffic.json")
    ap.add_argument("--kernel", default=None,
                    help="with --pmc-summary: the kernel (bench name); default: the roofline kernel "
                         "of the workload's last bench line in FETCH_DIR/bench.json")
    return ap.parse_args()


def log(msg):
    print("[bench] " + msg, file=sys.stderr, flush=True)


def measure_h2d_peak(torch, sizes=(64 << 20, 256 << 20), reps=8):
    """Best sustained pinned host -> device copy rate (GB/s) over large copies,
    using the same runtime call as the engine (hipMemcpyAsync via torch)."""
    best = 0.0
    n_max = max(sizes)
    h = torch.empty(n_max, dtype=torch.uint8, pin_memory=True)
    h.fill_(1)
    d = torch.empty(n_max, dtype=torch.uint8, device="cuda")
    s = torch.cuda.current_stream()
    for n in sizes:
        for _ in range(2):
            d[:n].copy_(h[:n], non_blocking=True)
        torch.cuda.synchronize()
        rates = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(s)
            d[:n].copy_(h[:n], non_blocking=True)
            e1.record(s)
            e1.synchronize()
            rates.append(n / (e0.elapsed_time(e1) * 1e-3) / 1e9)
        best = max(best, float(np.median(rates)))
    del h, d
    return best


def link_sweep(torch, reps=20):
    """Pinned host -> device copy rate by size, 4 KiB .. 1 GiB: median of
    `reps` timed copies (hipMemcpyAsync via torch, HIP events)."""
    n_max = 1 << 30
    h = torch.empty(n_max, dtype=torch.uint8, pin_memory=True)
    h.fill_(1)
    d = torch.empty(n_max, dtype=torch.uint8, device="cuda")
    s = torch.cuda.current_stream()
    n = 4 << 10
    while n <= n_max:
        for _ in range(2):
            d[:n].copy_(h[:n], non_blocking=True)
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(s)
            d[:n].copy_(h[:n], non_blocking=True)
            e1.record(s)
            e1.synchronize()
            ts.append(e0.elapsed_time(e1))
        ms = float(np.median(ts))
        print(json.dumps({"bytes": n, "median_ms": round(ms, 5), "gbps": round(n / (ms * 1e-3) / 1e9, 2),
                          "sdma": os.environ.get("HSA_ENABLE_SDMA", "default")}), flush=True)
        n *= 4
    del h, d


def measure_copy_chain(torch, sizes, reps=5):
    """Time (ms) of the swap-in copies alone: one pinned host -> device copy
    per slab, back to back on one stream with an event after each (as the
    engine issues them), no compute.  The floor that per-copy DMA start-up
    puts on a swapped inference with this many slabs."""
    total = sum(sizes)
    h = torch.empty(total, dtype=torch.uint8, pin_memory=True)
    h.fill_(1)
    d = torch.empty(total, dtype=torch.uint8, device="cuda")
    s = torch.cuda.Stream()
    evs = [torch.cuda.Event() for _ in sizes]
    best = None
    with torch.cuda.stream(s):
        for _ in range(reps + 1):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(s)
            off = 0
            for n, ev in zip(sizes, evs):
                d[off:off + n].copy_(h[off:off + n], non_blocking=True)
                ev.record(s)
                off += n
            e1.record(s)
            e1.synchronize()
            t = e0.elapsed_time(e1)
            best = t if best is None else min(best, t)
    del h, d
    return best


PARTITIONS = ("workload blocks", "balanced", "searched (delay model)")


def partition_name(choice, tuned):
    if tuned is None:
        return PARTITIONS[choice]
    best = min((t, i) for i, t in enumerate(tuned) if t)[1]
    return "tuned: " + PARTITIONS[best]


def quiet_gc():
    """Collect now and move every live object out of the collector's reach:
    a full collection of this process's objects (torch, numpy, weights)
    pauses the Python thread for several milliseconds, which would stall the
    enqueue of whichever inference it lands in."""
    gc.collect()
    gc.freeze()


def timed_loop(torch, eng, xd, yd, steps, warmup):
    quiet_gc()
    s = torch.cuda.current_stream()
    for _ in range(warmup):
        eng.infer_dev(xd.data_ptr(), yd.data_ptr(), s.cuda_stream)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(s)
    for _ in range(steps):
        eng.infer_dev(xd.data_ptr(), yd.data_ptr(), s.cuda_stream)
    e1.record(s)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) * 1e3
    return e0.elapsed_time(e1) / steps, wall / steps


def host_enqueue_us(torch, eng, xd, yd, n=10):
    """Host time of one sn_infer_dev call (the enqueue only), GPU idle."""
    s = torch.cuda.current_stream()
    ts = []
    for _ in range(n):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        eng.infer_dev(xd.data_ptr(), yd.data_ptr(), s.cuda_stream)
        ts.append((time.perf_counter() - t0) * 1e6)
    torch.cuda.synchronize()
    return float(np.median(ts))


def single_latency(torch, eng, xd, yd, n=10):
    """Latency of one isolated inference (no overlap with the previous one)."""
    s = torch.cuda.current_stream()
    ts = []
    for _ in range(n):
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(s)
        eng.infer_dev(xd.data_ptr(), yd.data_ptr(), s.cuda_stream)
        e1.record(s)
        e1.synchronize()
        ts.append(e0.elapsed_time(e1))
    return float(np.median(ts))


def recorded_traffic(kernel, workload):
    """HBM bytes per dispatch of `kernel` in `workload` from the committed
    counter summary (profiles/*_traffic.json), or None when there is none or
    the kernel source changed since the counters were taken."""
    import glob
    import hashlib
    src = os.path.join(ROOT, "paper_2401_16757_amd", "csrc", "kernels.hip")
    digest = hashlib.sha256(open(src, "rb").read()).hexdigest()
    for f in glob.glob(os.path.join(ROOT, "profiles", "*_traffic.json")):
        d = json.load(open(f))
        if d.get("kernel") == kernel and d.get("workload") == workload and \
                d.get("kernels_hip_sha256") == digest:
            return d["traffic_bytes_per_dispatch"]
    return None


def pmc_window(torch, eng, xd, yd):
    """Counter window: a 256 MiB device-to-device copy (its known bytes
    calibrate the counters and mark the start), PMC_INFERENCES all-resident
    inferences, then a 64 MiB copy (end marker).  The dispatches between the
    markers are one known set of whole inferences."""
    s = torch.cuda.current_stream()
    src = torch.empty(256 << 20, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    src.fill_(3)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    for _ in range(PMC_INFERENCES):
        eng.infer_dev(xd.data_ptr(), yd.data_ptr(), s.cuda_stream)
    torch.cuda.synchronize()
    dst[:64 << 20].copy_(src[:64 << 20])
    torch.cuda.synchronize()
    del src, dst


def kernel_symbol(name):
    """Demangled symbol of a conv kernel from its bench name."""
    import re
    m = re.match(r"conv3_mfma_(\d+)x(\d+)_s(\d+)_g(\d+)_(1x1|tap)$", name)
    if m:
        bm, bn, st, kg, kind = m.groups()
        return "void sn::conv_mfma3_kernel<%s, %s, %s, %d, %s>(sn::ConvArgs)" % (
            bm, bn, st, 0 if kind == "1x1" else 1, kg)
    m = re.match(r"conv_mfma_(\d+)x(\d+)x(\d+)_w(\d)(\d)_gen$", name)
    if m:
        return "void sn::conv_mfma_kernel<%s, %s, %s, %s, %s, false>(sn::ConvArgs)" % m.groups()
    raise ValueError("no symbol for kernel %r" % name)


def read_counters(d, counter):
    """Dispatches of a rocprofv3 --pmc CSV run: [(dispatch_id, kernel, value)]."""
    import csv
    import glob
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit("no *counter_collection.csv under %s" % d)
    rows = {}
    for f in files:
        for r in csv.DictReader(open(f)):
            if r["Counter_Name"] != counter:
                continue
            key = (f, int(r["Dispatch_Id"]))
            k = rows.setdefault(key, [r["Kernel_Name"], 0.0])
            k[1] += float(r["Counter_Value"])
    return [(key[1], v[0], v[1]) for key, v in sorted(rows.items())]


def window_average(rows, symbol, big_kib):
    """Average counter value per dispatch of `symbol` between the two marker
    copies, and the calibration copy's value (the first copy kernel whose
    count reaches big_kib / 4, then the next one past 1/16 of it)."""
    copies = [i for i, (_, k, v) in enumerate(rows) if "copyBuffer" in k and v >= big_kib / 4]
    if not copies:
        raise SystemExit("calibration copy not found")
    i0 = copies[0]
    cal = rows[i0][2]
    ends = [i for i, (_, k, v) in enumerate(rows) if i > i0 and "copyBuffer" in k and v >= cal / 16]
    if not ends:
        raise SystemExit("end marker not found")
    vals = [v for _, k, v in rows[i0 + 1:ends[0]] if k == symbol]
    if not vals:
        raise SystemExit("no dispatch of %s between the markers" % symbol)
    return sum(vals) / len(vals), len(vals), cal


def pmc_summary(a):
    """Traffic of one kernel from two counter runs, scaled by the counters'
    reading of the 256 MiB calibration copy (262144 KiB read and written)."""
    import hashlib
    fetch_dir, write_dir = a.pmc_summary
    kernel = a.kernel
    if kernel is None:
        bj = json.load(open(os.path.join(fetch_dir, "bench.json")))
        kernel = bj["roofline"]["kernel"]
    sym = kernel_symbol(kernel)
    ref_kib = 256 * 1024
    f_avg, n, f_cal = window_average(read_counters(fetch_dir, "FETCH_SIZE"), sym, ref_kib)
    w_avg, n2, w_cal = window_average(read_counters(write_dir, "WRITE_SIZE"), sym, ref_kib)
    fs, ws = ref_kib / f_cal, ref_kib / w_cal
    traffic = (f_avg * fs + w_avg * ws) * 1024
    src = os.path.join(ROOT, "paper_2401_16757_amd", "csrc", "kernels.hip")
    rec = {"kernel": kernel, "symbol": sym, "workload": a.workload,
           "fetch_kib_per_dispatch_raw": round(f_avg, 1), "write_kib_per_dispatch_raw": round(w_avg, 1),
           "dispatches": n, "inferences": PMC_INFERENCES,
           "fetch_scale": round(fs, 4), "write_scale": round(ws, 4),
           "traffic_bytes_per_dispatch": int(round(traffic)),
           "kernels_hip_sha256": hashlib.sha256(open(src, "rb").read()).hexdigest()}
    out = os.path.join(ROOT, "profiles", "%s_%s_traffic.json" % (kernel, a.workload))
    with open(out, "w") as fh:
        json.dump(rec, fh, indent=1)
    print(json.dumps(rec))
    print("wrote %s" % out, file=sys.stderr)


def conv_flops(spec, c0, c1):
    ho, wo = spec.out_hw()
    return 2.0 * ho * wo * (c1 - c0) * spec.c_in * spec.k * spec.k


def kernel_profile(S, net, eng, torch, xd, yd, reps=5):
    """Per-kernel times per inference of the swapped engine, the workload of
    the timed loop (timing level 2: every convolution launched with start /
    stop events of its own dispatch, a HIP event pair around every other
    layer piece), averaged over `reps` inferences and grouped by kernel.
    Returns {name: [launches, total_ms, flops, bytes]} per inference."""
    s = torch.cuda.current_stream()
    eng.set_option(S.OPT_TIMING, 2)
    for _ in range(2):
        eng.infer_dev(xd.data_ptr(), yd.data_ptr(), s.cuda_stream)
        torch.cuda.synchronize()
    # the per-piece events are read back by a host-API call
    x = xd.cpu().numpy()
    runs = []
    for _ in range(reps):
        eng.infer(x)
        runs.append(eng.pieces())
    eng.set_option(S.OPT_TIMING, 0)
    pieces = runs[0]
    for j, p in enumerate(pieces):
        p["t_ms"] = sum(r[j]["t_ms"] for r in runs) / reps
        p["t_main_ms"] = sum(r[j]["t_main_ms"] for r in runs) / reps
    groups = {}

    def add(name, t, fl, by):
        g = groups.setdefault(name, [0, 0.0, 0.0, 0.0])
        g[0] += 1
        g[1] += t
        g[2] += fl
        g[3] += by
    for p in pieces:
        spec = net.layers[p["layer"]]
        if spec.op == "conv2d":
            ho, wo = spec.out_hw()
            m, n = ho * wo, p["c1"] - p["c0"]
            # algorithmic bytes: input activation, weights, bias, output (and
            # residual) once each
            cin_p = (spec.c_in + 7) // 8 * 8
            act = spec.h_in * spec.w_in * cin_p * 2 + m * n * 2 * (2 if spec.res >= 0 else 1)
            add(S.kernel_name(p["kernel"]), p["t_main_ms"], conv_flops(spec, p["c0"], p["c1"]),
                p["w_bytes"] + p["b_bytes"] + act)
            if p["ksplit"] > 1:
                add("splitk_reduce", p["t_ms"] - p["t_main_ms"], 0.0,
                    4.0 * p["ksplit"] * m * n + 2.0 * m * n)
        elif spec.op == "linear":
            add("gemv", p["t_ms"], 2.0 * (p["c1"] - p["c0"]) * spec.c_in,
                p["w_bytes"] + p["b_bytes"] + 2 * spec.c_in + 2 * (p["c1"] - p["c0"]))
        else:
            add(spec.op, p["t_ms"], 0.0, 0.0)
    return groups


def slab_timeline(S, eng, x):
    """DMA / compute intervals of each slab in one host-API inference."""
    eng.set_option(S.OPT_TIMING, 1)
    eng.infer(x)
    eng.set_option(S.OPT_TIMING, 0)
    sl = eng.slabs()
    dma = [(s["t_in_start_ms"], s["t_in_start_ms"] + s["t_in_ms"]) for s in sl]
    comp = [(s["t_ex_start_ms"], s["t_ex_start_ms"] + s["t_ex_ms"]) for s in sl]
    dma_total = sum(b - a for a, b in dma)
    inter = 0.0
    for a, b in dma:
        for c, d in comp:
            inter += max(0.0, min(b, d) - max(a, c))
    return {"dma_ms": round(dma_total, 4), "compute_ms": round(sum(b - a for a, b in comp), 4),
            "overlap_frac": round(inter / dma_total, 4) if dma_total > 0 else None,
            "per_slab": [{"bytes": s["bytes"], "t_in_ms": round(s["t_in_ms"], 4),
                          "t_ex_ms": round(s["t_ex_ms"], 4),
                          "dma_gbs": round(s["bytes"] / (s["t_in_ms"] * 1e6), 2)
                          if s["t_in_ms"] > 0 else None} for s in sl]}


def cpu_baseline(net, wts, x, seconds):
    import oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()
                       if i.get("user_api") == "blas"] or [1])
    except Exception:
        threads = os.cpu_count()
    t0 = time.perf_counter()
    n = 0
    while True:
        oracle.forward(net, wts, x)
        n += 1
        el = time.perf_counter() - t0
        if el >= seconds or n >= 200:
            break
    return {"value": round(el / n * 1e3, 3), "unit": "ms/inference", "cores": int(threads),
            "kind": "oracle",
            "sample": "%d fp64 forward passes of %s (%.1f s) on host BLAS threads"
                      % (n, net.name, el)}



def direct_read_rate(path, reps=5):
    """Median rate (GB/s) of reading the whole image file as the engine does:
    one O_DIRECT read per slab (offsets and sizes from the file's header),
    the page cache bypassed, no GPU work alongside."""
    import mmap
    import statistics
    import struct
    head = open(path, "rb").read(4096)
    n = struct.unpack_from("<I", head, 12)[0]
    hb = struct.unpack_from("<Q", head, 24)[0]
    head = open(path, "rb").read(hb)
    reqs = []
    for i in range(n):
        _, nbytes, off, _ = struct.unpack_from("<QQQQ", head, 32 + 32 * i)
        reqs.append((off, (nbytes + 4095) // 4096 * 4096))
    buf = mmap.mmap(-1, max(r[1] for r in reqs))
    rates = []
    for _ in range(reps):
        try:
            fd = os.open(path, os.O_RDONLY | os.O_DIRECT)
        except OSError:
            fd = os.open(path, os.O_RDONLY)
        t0 = time.perf_counter()
        total = 0
        for off, ln in reqs:
            total += os.preadv(fd, [memoryview(buf)[:ln]], off)
        rates.append(total / (time.perf_counter() - t0) / 1e9)
        os.close(fd)
    buf.close()
    return statistics.median(rates)


def bench_storage(a, torch, S, net, wts, x, budget, frac_txt):
    """Storage tier (direct block fetch): the swapped plan's image in a file,
    every swap-in an O_DIRECT read into a pinned staging slot, then one DMA.
    One step = one inference; the bound is the storage read rate."""
    eng = S.build_engine(net, wts, budget=budget)
    tuned = eng.tune(5) if a.partition == 3 else None
    st = eng.stats()
    eng_res = S.build_engine(net, wts, budget=st["image_bytes"] + 4096)
    xd = torch.from_numpy(x).cuda()
    yd = torch.empty(eng.out_shape, dtype=torch.float16, device="cuda")
    yr = torch.empty(eng.out_shape, dtype=torch.float16, device="cuda")
    log("host-memory swapped reference")
    mem_ms, _ = timed_loop(torch, eng, xd, yd, a.steps, a.warmup)
    y_mem = yd.clone()
    log("writing the image file %s" % a.image_file)
    eng.save_image(a.image_file)
    raw_before = direct_read_rate(a.image_file)
    eng.attach_image_file(a.image_file)
    st2 = eng.stats()
    log("timing %d swapped steps from the file" % a.steps)
    r0 = st2["read_ms"]
    sw_ms, sw_wall = timed_loop(torch, eng, xd, yd, a.steps, a.warmup)
    read_ms = (eng.stats()["read_ms"] - r0) / (a.steps + a.warmup)
    res_ms, _ = timed_loop(torch, eng_res, xd, yr, a.steps, a.warmup)
    torch.cuda.synchronize()
    # the disk's sustained rate: a read burst right after the file was
    # written runs faster than the same reads a few seconds later
    raw = direct_read_rate(a.image_file)
    bitwise = bool(torch.equal(yd.view(torch.int16), yr.view(torch.int16))) and \
        bool(torch.equal(yd.view(torch.int16), y_mem.view(torch.int16)))
    streamed = st["streamed_bytes"]
    rate = streamed / (sw_ms * 1e-3) / 1e9
    out = {
        "metric": METRIC, "value": round(sw_ms / res_ms, 4), "unit": "x (swapped/resident latency)",
        "n_gpus": 1, "steps": a.steps, "warmup": a.warmup, "ms_per_step": round(sw_ms, 4),
        "higher_is_better": False, "scaling": "weak", "vs_baseline": None,
        "dtype": "f16 (fp32 accumulate)",
        "data": "synthetic (seeded He-normal weights, folded BN, N(0,1) input)",
        "config": {"workload": net.name, "batch": 1, "input": "x".join(map(str, net.input_shape)),
                   "weight_bytes": net.weight_bytes(), "budget_bytes": budget,
                   "budget_fraction": frac_txt, "slabs": st["n_slabs"],
                   "partition": partition_name(a.partition if a.partition < 3 else 0, tuned),
                   "weights": "image file, direct I/O" if st2["direct_io"] else "image file, buffered",
                   "parallelism": "none (1 GPU)"},
        "swapped_ms": round(sw_ms, 4), "resident_ms": round(res_ms, 4),
        "swapped_from_host_memory_ms": round(mem_ms, 4), "swapped_wall_ms": round(sw_wall, 4),
        "streamed_bytes_per_step": streamed,
        "storage": {"bound": "storage_read", "achieved": round(rate, 3), "peak": round(raw, 3),
                    "unit": "GB/s", "frac": round(rate / raw, 4) if raw > 0 else None,
                    "peak_right_after_write": round(raw_before, 3),
                    "read_ms_per_step": round(read_ms, 4)},
        "host_weight_bytes": st2["host_weight_bytes"], "image_bytes": st["image_bytes"],
        "direct_io": bool(st2["direct_io"]),
        "swapped_equals_resident_bitwise": bitwise,
    }
    eng.close()
    eng_res.close()
    print(json.dumps(out), flush=True)


def build_decoder(S, W, net, budget):
    """Register the decoder block by block, generating each block's weights
    just before it is added (the 13.5 GB of fp16 weights never coexist with
    a second full copy on the Python side)."""
    eng = S.SwapNet(budget)
    for a_, b_ in net.blocks:
        params = W.layers_params(net, range(a_, b_))
        descs, blob = S.block_payload(net, lambda li: params[li], a_, b_)
        eng.add_block(descs, blob)
        del params, blob
    eng.plan()
    eng.out_shape, eng.out_dtype = S.output_shape(net)
    return eng


def run_decoder(eng, prompt, gen):
    """Greedy generation: prefill, then gen-1 single-token steps.  Returns
    (prefill_ms, per-step ms list, token ids)."""
    eng.reset()
    quiet_gc()
    t0 = time.perf_counter()
    logits = eng.infer_tokens(prompt)
    pre = (time.perf_counter() - t0) * 1e3
    steps, ids = [], []
    for _ in range(gen - 1):
        nxt = int(np.argmax(logits))
        ids.append(nxt)
        t0 = time.perf_counter()
        logits = eng.infer_tokens(np.array([nxt], np.int32))
        steps.append((time.perf_counter() - t0) * 1e3)
    return pre, steps, ids


def bench_decoder(a, torch, S, W):
    net = W.get_network("decoder7b")
    gen = a.gen_tokens or net.extra["gen"]
    prompt = W.make_input(net)
    budget = net.budget_bytes()
    log("building swapped decoder (budget %d B = 4 layers)" % budget)
    eng = build_decoder(S, W, net, budget)
    eng.set_option(S.OPT_SYNC, a.sync)
    st = eng.stats()
    log("timing prefill + %d decode steps (swapped)" % (gen - 1))
    run_decoder(eng, prompt[:8], 3)                      # warm-up
    pre, steps, ids = run_decoder(eng, prompt, gen)
    eng.close()
    log("building resident decoder")
    eng_r = build_decoder(S, W, net, st["image_bytes"] + (1 << 20))
    run_decoder(eng_r, prompt[:8], 3)
    pre_r, steps_r, ids_r = run_decoder(eng_r, prompt, gen)
    eng_r.close()
    peak = measure_h2d_peak(torch)
    dec = float(np.median(steps))
    dec_r = float(np.median(steps_r))
    streamed = st["streamed_bytes"] + 2 * net.extra["d"]   # + one embedding row
    out = {
        "metric": METRIC, "value": round(dec / dec_r, 3), "unit": "x (swapped/resident decode latency)",
        "n_gpus": 1, "steps": gen - 1, "warmup": 2, "ms_per_step": round(dec, 3),
        "higher_is_better": False, "scaling": "weak", "vs_baseline": None,
        "dtype": "f16 (fp32 accumulate)", "data": "synthetic (seeded N(0,0.02) weights, random prompt)",
        "config": {"workload": "decoder7b", "batch": 1, "prompt": len(prompt), "generated": gen,
                   "weight_bytes": net.weight_bytes(), "budget_bytes": budget,
                   "budget_fraction": "4 layers", "slabs": st["n_slabs"],
                   "parallelism": "none (1 GPU)"},
        "prefill_ms": round(pre, 2), "resident_prefill_ms": round(pre_r, 2),
        "decode_ms_per_token": round(dec, 3), "resident_decode_ms_per_token": round(dec_r, 3),
        "decode_tokens_per_s": round(1e3 / dec, 3),
        "streamed_bytes_per_token": streamed,
        "h2d_gbps": round(streamed / (dec * 1e-3) / 1e9, 2), "h2d_peak_gbps": round(peak, 2),
        "h2d_frac": round(streamed / (dec * 1e-3) / 1e9 / peak, 4),
        "link": {"bound": "pcie_h2d", "achieved": round(streamed / (dec * 1e-3) / 1e9, 2),
                 "peak": round(peak, 2), "unit": "GB/s",
                 "frac": round(streamed / (dec * 1e-3) / 1e9 / peak, 4), "traffic": streamed},
        "resident_hbm_gbps": round(streamed / (dec_r * 1e-3) / 1e9, 1),
        "same_tokens_swapped_and_resident": ids == ids_r,
        "kv_bytes": st["kv_bytes"], "swapin_mode": "SDMA, copy thread",
    }
    print(json.dumps(out), flush=True)


def main():
    a = parse()
    if a.pmc_summary:
        return pmc_summary(a)
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if a.gpus != 1 or world != 1:
        print("bench.py: this engine runs on one GPU; --gpus %d is not supported "
              "(multi-GPU sharding is a design note only)" % a.gpus, file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2401_16757_amd import swapnet as S
    from paper_2401_16757_amd import workloads as W

    torch.cuda.set_device(0)
    # all engine work goes to a non-default stream, so that torch's events
    # (recorded on the current stream) bracket it
    stream = torch.cuda.Stream()
    torch.cuda.set_stream(stream)
    if a.link_sweep:
        return link_sweep(torch)
    if a.workload == "decoder7b":
        return bench_decoder(a, torch, S, W)
    net = W.get_network(a.workload)
    log("generating %s weights" % net.name)
    wts = W.make_weights(net)
    x = W.make_input(net)
    budget = net.budget_bytes() if a.budget_frac is None else int(net.weight_bytes() * a.budget_frac)
    frac_txt = {"resnet50": "1/2.32", "vgg16": "1/5.81", "fcn_resnet101": "1/3",
                "tiny_cnn": "0.6"}[net.name] if a.budget_frac is None else "%.4f" % a.budget_frac

    if a.image_file:
        return bench_storage(a, torch, S, net, wts, x, budget, frac_txt)
    cm = None
    if a.partition == 2:
        log("calibrating the delay model on the workload-block plan")
        with S.build_engine(net, wts, budget=budget) as cal:
            cal.set_option(S.OPT_COPY_STREAMS, a.copy_streams)
            cal.calibrate(5)
            cm = cal.cost_model()
    log("planning swapped engine (budget %d B) and resident engine" % budget)
    eng_sw = S.build_engine(net, wts, budget=budget, partition=min(a.partition, 2), cost_model=cm)
    # DMA queue use before the partition is chosen: it changes the per-DMA cost
    eng_sw.set_option(S.OPT_COPY_STREAMS, a.copy_streams)
    tuned = None
    if a.partition == 3:
        log("choosing the partition by measurement (untimed)")
        tuned = eng_sw.tune(5)
        cm = eng_sw.cost_model()
    st = eng_sw.stats()
    eng_res = S.build_engine(net, wts, budget=st["image_bytes"] + 4096)
    eng_sw.set_option(S.OPT_SWAPIN, a.swapin)
    eng_sw.set_option(S.OPT_COPY_STREAMS, a.copy_streams)
    eng_sw.set_option(S.OPT_SYNC, a.sync)
    if a.swapin_blocks:
        eng_sw.set_option(S.OPT_SWAPIN_BLOCKS, a.swapin_blocks)
    if a.no_graph:
        eng_sw.set_option(S.OPT_GRAPH, 0)
        eng_res.set_option(S.OPT_GRAPH, 0)
    assert eng_res.stats()["resident"] == 1 and st["resident"] == 0

    xd = torch.from_numpy(x).cuda()
    yd = torch.empty(eng_sw.out_shape, dtype=torch.float16, device="cuda")
    yr = torch.empty(eng_sw.out_shape, dtype=torch.float16, device="cuda")

    log("measuring pinned H2D peak")
    peak = measure_h2d_peak(torch)

    log("timing %d swapped steps" % a.steps)
    sw_ms, sw_wall = timed_loop(torch, eng_sw, xd, yd, a.steps, a.warmup)
    log("timing %d resident steps" % a.steps)
    res_ms, res_wall = timed_loop(torch, eng_res, xd, yr, a.steps, a.warmup)
    sw_lat = single_latency(torch, eng_sw, xd, yd)
    res_lat = single_latency(torch, eng_res, xd, yr)
    sw_host = host_enqueue_us(torch, eng_sw, xd, yd)
    res_host = host_enqueue_us(torch, eng_res, xd, yr)
    torch.cuda.synchronize()
    bitwise = bool(torch.equal(yd.view(torch.int16), yr.view(torch.int16)))

    ablation = None
    if a.ablation:
        # the redundant memory operations of plain swapping, put back one at
        # a time (sequential = swap-in then compute, slab after slab)
        ablation = {}
        for name, flags in (("sequential", 1), ("sequential + hipMalloc/hipFree per swap", 3),
                            ("sequential + pageable source", 5),
                            ("sequential + copy-based assembly", 9), ("all three", 15)):
            log("ablation: %s" % name)
            eng_sw.set_option(S.OPT_NAIVE, flags)
            ablation[name] = round(timed_loop(torch, eng_sw, xd, yd, 10, 2)[0], 4)
        eng_sw.set_option(S.OPT_NAIVE, 0)

    streamed = st["streamed_bytes"]
    h2d = streamed / (sw_ms * 1e-3) / 1e9
    log("timing the swap-in copies alone")
    chain_ms = measure_copy_chain(torch, [sl["bytes"] for sl in eng_sw.slabs()])
    log("timeline and kernel profile (untimed passes)")
    tl = slab_timeline(S, eng_sw, x)
    if cm is None:
        # the delay model of this plan, measured on it (for the prediction)
        eng_sw.calibrate(5)
    model = eng_sw.cost_model()
    pred_lat, pred_per = eng_sw.predict()
    groups = kernel_profile(S, net, eng_sw, torch, xd, yd)
    conv = {k: v for k, v in groups.items() if k.startswith("conv")}
    dom = max(conv.items(), key=lambda kv: kv[1][1]) if conv else None
    total_flops = sum(v[2] for v in groups.values())
    res_compute_ms = sum(v[1] for v in groups.values())
    roofline = None
    if dom:
        # the kernel's bound: MFMA if its FLOPs take longer at peak than its
        # algorithmic bytes at HBM peak, else HBM (batch-1 layers mostly are)
        name, (launches, tms, fl, by) = dom
        if fl / (MFMA_FP16_PEAK_TFLOPS * 1e12) >= by / (HBM_PEAK_GBS * 1e9):
            ach, peak_r, unit, bound = fl / (tms * 1e-3) / 1e12, MFMA_FP16_PEAK_TFLOPS, "TFLOP/s", "mfma"
        else:
            ach, peak_r, unit, bound = by / (tms * 1e-3) / 1e9, HBM_PEAK_GBS, "GB/s", "hbm"
        roofline = {"bound": bound, "kernel": name, "launches_per_step": launches,
                    "avg_launch_us": round(tms / launches * 1e3, 3),
                    "achieved": round(ach, 2), "peak": peak_r, "unit": unit,
                    "frac": round(ach / peak_r, 5),
                    "flops_per_launch": round(fl / launches), "bytes_per_launch": round(by / launches),
                    "mfma_tflops": round(fl / (tms * 1e-3) / 1e12, 2),
                    "traffic": recorded_traffic(name, a.workload)}
    mfma_util = (total_flops / (res_compute_ms * 1e-3) / 1e12) / MFMA_FP16_PEAK_TFLOPS \
        if res_compute_ms > 0 else None

    out = {
        "metric": METRIC,
        "value": round(sw_ms / res_ms, 4),
        "unit": "x (swapped/resident latency)",
        "n_gpus": 1, "steps": a.steps, "warmup": a.warmup,
        "ms_per_step": round(sw_ms, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16 (fp32 accumulate)",
        "data": "synthetic (seeded He-normal weights, folded BN, N(0,1) input)",
        "config": {"workload": net.name, "batch": 1, "input": "x".join(map(str, net.input_shape)),
                   "weight_bytes": net.weight_bytes(), "budget_bytes": budget,
                   "budget_fraction": frac_txt, "user_blocks": len(net.blocks),
                   "slabs": st["n_slabs"],
                   "partition": partition_name(a.partition, tuned),
                   "sync": ["events", "stream values", "rocr copies + gate kernels"][a.sync],
                   "parallelism": "none (1 GPU)"},
        "swapped_ms": round(sw_ms, 4), "resident_ms": round(res_ms, 4),
        "swapped_latency_ms": round(sw_lat, 4), "resident_latency_ms": round(res_lat, 4),
        "swapped_wall_ms": round(sw_wall, 4), "resident_wall_ms": round(res_wall, 4),
        "host_enqueue_us": {"swapped": round(sw_host, 1), "resident": round(res_host, 1)},
        "throughput_inf_per_s": round(1e3 / sw_ms, 2),
        "streamed_bytes_per_step": streamed,
        "h2d_gbps": round(h2d, 2), "h2d_peak_gbps": round(peak, 2),
        "h2d_frac": round(h2d / peak, 4),
        "link": {"bound": "pcie_h2d", "achieved": round(h2d, 2), "peak": round(peak, 2),
                 "unit": "GB/s", "frac": round(h2d / peak, 4),
                 "traffic": streamed,
                 "copy_chain_ms": round(chain_ms, 4),
                 "swapped_vs_copy_chain": round(chain_ms / sw_ms, 4)},
        "link_floor_ms": round(streamed / (peak * 1e9) * 1e3, 4),
        "mfma_util": round(mfma_util, 5) if mfma_util else None,
        "roofline": roofline,
        "timeline": {k: v for k, v in tl.items() if k != "per_slab" or a.verbose},
        "delay_model": {"link_gbps": round(1e-9 / model["alpha"], 2) if model["alpha"] > 0 else None,
                        "beta_us": round(model["beta"] * 1e6, 2),
                        "gate_us": round(model["gate"] * 1e6, 2),
                        "wake_us": round(model["wake"] * 1e6, 2),
                        "slab_ex_us": round(model["slab_ex"] * 1e6, 2),
                        "predicted_latency_ms": round(pred_lat * 1e3, 4),
                        "predicted_ms_per_step": round(pred_per * 1e3, 4),
                        "calibrated_on": "this plan" if cm is None else "workload-block plan"},
        "kernels": {k: {"launches": v[0], "ms": round(v[1], 4)} for k, v in groups.items()},
        "swapped_equals_resident_bitwise": bitwise,
        "ablation_ms": ablation,
        "partition_candidates_ms": None if tuned is None else
            {n: round(t * 1e3, 4) if t else None for n, t in zip(PARTITIONS, tuned)},
        "activation_bytes": st["activation_bytes"],
        "hip_graph": not a.no_graph,
        "swapin_mode": {0: "copy kernel", 1: "SDMA, calling thread", 2: "SDMA, copy thread"}[a.swapin],
    }
    # runtime adaptation (Sec. 6): re-plan in place for half the budget and
    # back, with the workload's blocks (host wall time of each sn_replan)
    eng_sw.set_option(S.OPT_PARTITION, 0)
    t0 = time.perf_counter()
    eng_sw.replan(budget // 2)
    t1 = time.perf_counter()
    eng_sw.replan(budget)
    t2 = time.perf_counter()
    out["replan_ms"] = {"to_half_budget": round((t1 - t0) * 1e3, 2), "back": round((t2 - t1) * 1e3, 2)}
    if a.pmc_calibration:
        pmc_window(torch, eng_res, xd, yr)
    if not a.no_cpu_baseline:
        log("CPU oracle baseline (~%.0f s)" % a.cpu_seconds)
        out["cpu_baseline"] = cpu_baseline(net, wts, x, a.cpu_seconds)
    eng_sw.close()
    eng_res.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

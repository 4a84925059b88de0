"""Benchmark: images/s of one CNN partition forward on one MI355X.

Default workload: ResNet-152, the whole model (158 fused layers, stem to
softmax), fp16, batch 64 on 64 x 3 x 224 x 224 seeded synthetic images with
seeded He-init weights: the largest batch of the 1..64 range whose per-layer
latency table the paper's planner consumes (Sec. 5.1; App. A.1, L_kbi).  A
step is one forward of the whole range at that batch, inputs resident in
HBM.  Other workloads: --workload NAME [--batch B].  Prints one JSON line with the
throughput, the roofline position of the dominant kernel (per-launch HIP
event timing on the stream the kernels run on) and the CPU oracle timed on
a bounded sample as a baseline.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "CNN-partition images/sec at batch 1–64; per-layer MFMA % or HBM GB/s"
PEAK_MFMA_TFLOPS = {"f16": 2516.6, "bf16": 2516.6, "f32": 157.3}
PEAK_HBM_GBS = 8000.0
DTYPE_LABEL = {"f32": "f32", "f16": "f16", "bf16": "bf16"}
DEFAULT_WORKLOAD = "resnet152"
DEFAULT_BATCH = {"resnet152": 64}


def roofline(records, dtype):
    """Dominant kernel (largest total time per step) and its position."""
    groups = {}
    for r in records:
        g = groups.setdefault(r["kernel"], {"us": 0.0, "flops": 0.0, "bytes": 0.0, "n": 0})
        g["us"] += r["mean_us"]
        g["flops"] += r["flops"]
        g["bytes"] += r["bytes"]
        g["n"] += 1
    name, g = max(groups.items(), key=lambda kv: kv[1]["us"])
    t_mfma = g["flops"] / (PEAK_MFMA_TFLOPS[dtype] * 1e12)
    t_hbm = g["bytes"] / (PEAK_HBM_GBS * 1e9)
    avg_us = g["us"] / g["n"]
    if t_mfma >= t_hbm:
        achieved = g["flops"] / g["n"] / (avg_us * 1e-6) / 1e12
        out = {"bound": "mfma", "achieved": achieved, "peak": PEAK_MFMA_TFLOPS[dtype],
               "unit": "TFLOP/s"}
    else:
        achieved = g["bytes"] / g["n"] / (avg_us * 1e-6) / 1e9
        out = {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s"}
    out["frac"] = out["achieved"] / out["peak"]
    out["traffic"] = None   # filled from committed HBM counters, see measured_traffic
    out["kernel"] = name
    out["launches_per_step"] = g["n"]
    out["algorithmic_bytes_per_launch"] = g["bytes"] / g["n"]
    out["algorithmic_flops_per_launch"] = g["flops"] / g["n"]
    out["avg_launch_us"] = avg_us
    out["share_of_step"] = g["us"] / sum(v["us"] for v in groups.values())
    return out


def cold_summary(records, dtype, copy_fit=None):
    """Roofline fractions from isolated-cold launches (caches swept before
    every repetition): per kernel family, HBM fraction bytes-weighted
    (sum of bytes / (peak x sum of time)) for memory-bound families and for
    GEMM launches the roofline puts on HBM, MFMA fraction FLOP-weighted for
    GEMM launches it puts on MFMA.  Launches moving < 16 MB are counted
    separately as launch-bound.  With a cold-copy fit (copy_reference), each
    memory-bound family also reports, over its launches of at least 16 MB,
    the time a plain device copy of the same bytes takes under the same
    isolated-cold method, summed, over the family's time."""
    peak_f = PEAK_MFMA_TFLOPS[dtype] * 1e12
    peak_b = PEAK_HBM_GBS * 1e9
    fam = {}
    for r in records:
        name = r["kernel"].split("<")[0]
        t = r["median_us"] * 1e-6
        if name.startswith("conv_gemm"):
            if r["flops"] / peak_f >= r["bytes"] / peak_b:
                name = "conv_gemm (MFMA-bound launches)"
            else:
                name = "conv_gemm (HBM-bound launches)"
        g = fam.setdefault(name, {"us": 0.0, "bytes": 0.0, "flops": 0.0, "launches": 0,
                                  "small_launches": 0, "us_big": 0.0, "bytes_big": 0.0,
                                  "copy_us_big": 0.0})
        g["us"] += r["median_us"]
        g["bytes"] += r["bytes"]
        g["flops"] += r["flops"]
        g["launches"] += 1
        if r["bytes"] < 16e6:
            g["small_launches"] += 1
        else:
            g["us_big"] += r["median_us"]
            g["bytes_big"] += r["bytes"]
            if copy_fit:
                g["copy_us_big"] += copy_fit["t0_us"] + r["bytes"] / (copy_fit["gb_per_s"] * 1e3)
    out = {}
    for name, g in fam.items():
        if g["us"] <= 0:
            continue
        d = {"us_per_step": round(g["us"], 2), "launches": g["launches"],
             "launches_under_16MB": g["small_launches"]}
        if "MFMA-bound" in name:
            d["mfma_frac"] = g["flops"] / (g["us"] * 1e-6 * peak_f)
        else:
            d["hbm_frac"] = g["bytes"] / (g["us"] * 1e-6 * peak_b)
            if g["us_big"] > 0:
                d["hbm_frac_launches_over_16MB"] = g["bytes_big"] / (g["us_big"] * 1e-6 * peak_b)
                if copy_fit:
                    d["vs_cold_copy_launches_over_16MB"] = g["copy_us_big"] / g["us_big"]
        out[name] = d
    return out


def launch_floor(n=200, reps=10):
    """Per-launch time of back-to-back dependent kernels replayed from one
    captured graph: n in-place adds on one element (a 1-block kernel that
    loads and stores), and on 1 MiB (1024 blocks).  The floor every launch of
    a partition pays before its own work."""
    import torch
    out = {"launches_per_graph": n}
    for label, numel in (("1 element", 1), ("1 MiB", 1 << 18)):
        x = torch.zeros(numel, dtype=torch.float32, device="cuda")
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            for _ in range(3):
                x.add_(1.0)
        torch.cuda.current_stream().wait_stream(s)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(n):
                x.add_(1.0)
        for _ in range(5):
            g.replay()
        torch.cuda.synchronize()
        best = 1e9
        for _ in range(reps):
            t0 = time.perf_counter()
            g.replay()
            torch.cuda.synchronize()
            best = min(best, time.perf_counter() - t0)
        out[f"us_per_launch_{label.replace(' ', '_')}"] = best * 1e6 / n
    return out


def copy_reference(sizes_mb=(8, 16, 32, 64, 128, 256), reps=5):
    """HBM fraction a plain device copy reaches under the isolated-cold
    method (a 1 GiB read sweep before each repetition, evicting L2 and the
    memory-side cache), and warm: the practical ceiling the memory-bound
    kernels' isolated-cold fractions compare with.  Bytes moved = read +
    write of the copy; median over `reps`."""
    import torch
    sweep = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
    out = {}
    for mb in sizes_mb:
        n = int(mb * 2 ** 20) // 8              # mb megabytes moved: half read, half written
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        res = {}
        for mode in ("cold", "warm"):
            ts = []
            for _ in range(reps):
                if mode == "cold":
                    _ = sweep.sum()
                else:
                    dst.copy_(src)
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                dst.copy_(src)
                e1.record()
                torch.cuda.synchronize()
                ts.append(e0.elapsed_time(e1) * 1e-3)
            t = sorted(ts)[len(ts) // 2]
            res[f"{mode}_us"] = round(t * 1e6, 2)
            res[f"{mode}_hbm_frac"] = 2 * n * 4 / t / (PEAK_HBM_GBS * 1e9)
        out[f"{mb}MB"] = res
        del src, dst
    del sweep
    torch.cuda.synchronize()
    # least-squares fit of the cold copy time, t = t0 + bytes / bw, for the
    # per-family comparison in cold_summary
    xs = [float(k[:-2]) * 2 ** 20 for k in out]
    ys = [v["cold_us"] for v in out.values()]
    mx, my = sum(xs) / len(xs), sum(ys) / len(ys)
    slope = sum((x - mx) * (y - my) for x, y in zip(xs, ys)) / sum((x - mx) ** 2 for x in xs)
    out["cold_fit"] = {"t0_us": my - slope * mx, "gb_per_s": 1e-3 / slope}
    return out


def batch_sweep(part, max_batch, xd, out, stream, batches, steps=20, rounds=3):
    """Partition latency and images/s at several batches on the benchmark's
    handle: a graph captured per batch on the leading images of the same
    input and output buffers, best of `rounds` runs of `steps` replays."""
    import torch
    res = {"batches": [], "ms_per_step": [], "images_per_s": []}
    for b in batches:
        if b > max_batch:
            continue
        part.capture(b, xd.data_ptr(), out.data_ptr())
        for _ in range(5):
            part.run(b, xd.data_ptr(), out.data_ptr(), stream)
        torch.cuda.synchronize()
        best = 1e9
        for _ in range(rounds):
            t0 = time.perf_counter()
            for _ in range(steps):
                part.run(b, xd.data_ptr(), out.data_ptr(), stream)
            torch.cuda.synchronize()
            best = min(best, (time.perf_counter() - t0) / steps)
        res["batches"].append(b)
        res["ms_per_step"].append(round(best * 1e3, 4))
        res["images_per_s"].append(round(b / best, 1))
    res["method"] = (f"one captured graph per batch on the bench handle, best of {rounds} runs of "
                     f"{steps} back-to-back replays (wall clock)")
    return res


def write_table_json(path, out):
    """Writes a latency table compactly: per-batch lists aligned with
    out["batches"] (microseconds to 0.01, fractions to 4 digits), a layer's
    bound as one string when it is the same at every batch, one row a line."""
    def r(v, nd):
        return None if v is None else round(float(v), nd)
    head = {k: v for k, v in out.items() if k != "rows"}
    for k in ("partition_us", "sum_of_layers_us", "images_per_s"):
        head[k] = [r(v, 2) for v in head[k]]
    lines = []
    for row in out["rows"]:
        row = dict(row)
        row["us"] = [r(v, 2) for v in row["us"]]
        row["roofline_frac"] = [r(v, 4) for v in row["roofline_frac"]]
        if len(set(row["bound"])) == 1:
            row["bound"] = row["bound"][0]
        lines.append(json.dumps(row, separators=(",", ":")))
    text = ("{\n" + "".join(f" {json.dumps(k)}: {json.dumps(v, separators=(',', ':'))},\n"
                             for k, v in head.items())
            + ' "rows": [\n' + ",\n".join(lines) + "\n ]\n}\n")
    json.loads(text)
    with open(path, "w") as f:
        f.write(text)


def source_digest():
    """sha256 over the sources that define the GEMM kernel whose HBM counters
    are recorded and the planner that configures it (conv_gemm.hip,
    kernels.h, runtime.hip): a change to any of them invalidates counters
    taken before it."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2507_18748_amd", "csrc")
    for f in ("conv_gemm.hip", "kernels.h", "runtime.hip"):
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()


def _pmc_per_dispatch(csv_dir, counter, match):
    """Mean value of `counter` per dispatch of kernels whose name contains
    `match`, from a rocprofv3 --pmc csv directory (run_counter_collection.csv)."""
    import csv
    import glob
    vals = []
    for path in glob.glob(os.path.join(csv_dir, "**", "*counter_collection.csv"), recursive=True):
        with open(path) as f:
            for r in csv.DictReader(f):
                if r["Counter_Name"] == counter and match in r["Kernel_Name"]:
                    vals.append(float(r["Counter_Value"]))
    return (sum(vals) / len(vals), len(vals)) if vals else (None, 0)


def kernel_symbol(kernel):
    """Mangled-name prefix of a LDS-staged GEMM configuration name such as
    conv_gemm<f16,64x64,kv8,dma2> or conv_gemm_mx<bf16,128x128,4w,dma3>."""
    fam, rest = kernel.split("<", 1)
    parts = rest.rstrip(">").split(",")
    t = {"f16": "DF16_", "bf16": "DF16b", "f32": "f"}[parts[0]]
    bm, bn = (int(v) for v in parts[1].split("x"))
    waves = 4
    for q in parts[2:]:
        if q.endswith("w"):
            waves = int(q[:-1])
    ns = int([q for q in parts if q.startswith("dma")][0][3:])
    tapv = 1 if "tapv" in parts else 0
    if fam == "conv_gemm_mx":
        wm = {4: 2, 8: 4 if bm == 256 else 2}[waves]
        return f"conv_gemm_mxI{t}Li{bm}ELi{bn}ELi{wm}ELi{waves // wm}ELi{ns}ELb{tapv}E"
    wm, wn = {1: (1, 1), 2: (1, 2), 4: (2, 2), 8: (2, 4)}[waves]
    return f"conv_gemm_dmaI{t}Li{bm}ELi{bn}ELi{wm}ELi{wn}ELi{ns}ELb{tapv}E"


def traffic_record(args):
    """Writes the HBM-traffic record of the workload's dominant kernel from
    four rocprofv3 --pmc runs under --pmc-dir: FETCH_SIZE and WRITE_SIZE of
    the benchmark command, and of a plain device copy (--copy-calibration),
    in subdirectories FETCH_SIZE, WRITE_SIZE, copy_FETCH_SIZE,
    copy_WRITE_SIZE.  The copy's counters against its known size give the
    scale of each counter; the record carries the sha256 of the sources the
    counters describe, so bench.py reports them only while those hold."""
    rec_in = json.load(open(args.traffic_from))      # a bench.py line (--kernels run) of the same command
    roof = rec_in["roofline"]
    kernel = roof["kernel"]
    match = kernel_symbol(kernel)
    d = args.pmc_dir
    fetch, nf = _pmc_per_dispatch(os.path.join(d, "FETCH_SIZE"), "FETCH_SIZE", match)
    write, nw = _pmc_per_dispatch(os.path.join(d, "WRITE_SIZE"), "WRITE_SIZE", match)
    cf, _ = _pmc_per_dispatch(os.path.join(d, "copy_FETCH_SIZE"), "FETCH_SIZE", "copyBuffer")
    cw, _ = _pmc_per_dispatch(os.path.join(d, "copy_WRITE_SIZE"), "WRITE_SIZE", "copyBuffer")
    copy_kib = args.copy_mib * 1024.0
    fs, ws = copy_kib / cf, copy_kib / cw
    out = {"workload": rec_in["config"]["name"], "batch": rec_in["config"]["batch"], "kernel": kernel,
           "kernel_symbol_match": match,
           "source_sha256": source_digest(),
           "fetch_kib_per_dispatch": fetch, "write_kib_per_dispatch": write,
           "fetch_scale": fs, "write_scale": ws, "dispatches": [nf, nw],
           "traffic_bytes_per_launch": (fetch * fs + write * ws) * 1024.0,
           "algorithmic_bytes_per_launch": roof.get("algorithmic_bytes_per_launch"),
           "commands": args.pmc_commands.split(";") if args.pmc_commands else [],
           "note": "FETCH_SIZE and WRITE_SIZE in KiB per dispatch of the dominant kernel's "
                   "configuration, mean over every dispatch of the profiled command; scaled by "
                   "a plain device copy's counters (reads x fetch_scale, writes x write_scale); "
                   "bench.py reports traffic only while source_sha256 matches conv_gemm.hip, "
                   "kernels.h and runtime.hip"}
    with open(args.traffic_record, "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps(out))


def measured_traffic(workload, kernel, batch=None):
    """HBM bytes per launch of `kernel` on `workload` from a committed counter
    record (profiles/*_traffic.json: FETCH_SIZE and WRITE_SIZE per dispatch,
    scaled by a plain copy's counters), or None when there is none or the
    sources changed since the counters were taken."""
    import glob
    digest = None
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*_traffic.json"))):
        with open(path) as f:
            rec = json.load(f)
        if rec.get("workload") != workload or rec.get("kernel") != kernel:
            continue
        if batch is not None and rec.get("batch", batch) != batch:
            continue
        digest = digest or source_digest()
        if rec.get("source_sha256") == digest:
            return rec["traffic_bytes_per_launch"]
    return None


def host_cpu():
    """Host facts for the CPU baseline: logical CPUs, model name, OpenMP setting."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"nproc": os.cpu_count(), "affinity": len(os.sched_getaffinity(0)),
            "cpu_model": model, "OMP_NUM_THREADS": os.environ.get("OMP_NUM_THREADS")}


def cpu_baseline(wl, m, P, target_s, sample_batches=(1, 4)):
    """The oracle on a bounded sample of the workload: one pass at each of
    `sample_batches` (images of the same seeded input), then the last batch
    repeated until `target_s` of wall time.  images/s over the whole sample."""
    import oracle
    images, el, per = 0, 0.0, {}
    for b in sample_batches:
        x = wl.input(b)
        n = 0
        t0 = time.perf_counter()
        while True:
            oracle.forward(m.layers, P, wl.begin, wl.end, x, wl.dtype)
            n += b
            t = time.perf_counter() - t0
            if b != sample_batches[-1] or el + t >= target_s:
                break
        per[b] = n / t
        images += n
        el += t
    out = {"value": images / el, "unit": "images/s", "cores": oracle.num_threads(),
           "kind": "oracle",
           "sample": f"{images} images of the workload's seeded input: batch "
                     + ", then ".join(f"{b} ({per[b]:.2f} images/s)" for b in sample_batches)
                     + f" repeated; {el:.1f} s wall"}
    out.update(host_cpu())
    return out


def library_baseline(wl, m, P, x_nchw, steps, warmup, ref_out=None):
    """The same partition on PyTorch-ROCm's own kernels (MIOpen convolutions,
    BLAS linear layers, PyTorch's pooling and elementwise kernels): NHWC
    (channels_last) activations in the workload's dtype, batch norm folded
    into the convolution weights and bias in fp64 before the cast, the
    residual add and activation as separate elementwise ops, softmax in fp32.
    Timed eagerly and as one captured CUDA graph, inputs resident on the GPU.
    A measured comparison on the same hardware, not part of the path."""
    import numpy as np
    import torch
    import torch.nn.functional as F
    torch.backends.cudnn.benchmark = True
    tdt = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}[wl.dtype]
    cl = torch.channels_last
    layers = m.layers
    prm = {}
    for i in range(wl.begin, wl.end):
        L, p = layers[i], P[i]
        if L.op not in ("conv", "fc", "fc_softmax"):
            continue
        w = torch.from_numpy(p["weight"]).double()
        b = torch.from_numpy(p["bias"]).double() if "bias" in p else torch.zeros(L.c_out, dtype=torch.float64)
        if L.bn:
            sc = torch.from_numpy(p["bn_gamma"]).double() / torch.sqrt(
                torch.from_numpy(p["bn_var"]).double() + 1e-5)
            w = w * sc.reshape(-1, *([1] * (w.dim() - 1)))
            b = (b - torch.from_numpy(p["bn_mean"]).double()) * sc + torch.from_numpy(p["bn_beta"]).double()
        w = w.to(tdt).cuda()
        prm[i] = (w.contiguous(memory_format=cl) if w.dim() == 4 else w, b.to(tdt).cuda())

    def act(y, a):
        if a == "relu":
            return F.relu(y)
        if a == "relu6":
            return F.hardtanh(y, 0.0, 6.0)
        return y

    def fwd(x, progress=False):
        outs = {wl.begin - 1: x}
        last = time.perf_counter()
        for i in range(wl.begin, wl.end):
            if progress and time.perf_counter() - last > 10:
                torch.cuda.synchronize()
                print(f"[bench] library baseline first pass at layer {i}", file=sys.stderr,
                      flush=True)
                last = time.perf_counter()
            L = layers[i]
            h = outs[L.src]
            if L.op == "conv":
                y = F.conv2d(h, prm[i][0], prm[i][1], L.stride, L.pad, 1, L.groups)
                if L.res_src >= 0:
                    y = y + outs[L.res_src]
                y = act(y, L.act)
            elif L.op == "maxpool":
                y = F.max_pool2d(h, L.k, L.stride, L.pad)
            elif L.op == "gap":
                y = h.mean((2, 3), keepdim=True)
            else:
                y = act(F.linear(h.flatten(1), prm[i][0], prm[i][1]), L.act)
                if L.op == "fc_softmax":
                    y = torch.softmax(y.float(), 1)
            outs[i] = y
        return outs[wl.end - 1]

    x = torch.from_numpy(np.ascontiguousarray(x_nchw)).to(tdt).cuda().contiguous(memory_format=cl)
    t0 = time.perf_counter()
    with torch.no_grad():
        y_eager = fwd(x, progress=True)
        for _ in range(max(warmup, 3)):
            y_eager = fwd(x)
        torch.cuda.synchronize()
        print(f"[bench] library baseline warmup {time.perf_counter() - t0:.1f} s",
              file=sys.stderr, flush=True)
        t0 = time.perf_counter()
        for _ in range(steps):
            fwd(x)
        torch.cuda.synchronize()
        eager_s = time.perf_counter() - t0
        res = {"kind": "pytorch-rocm " + torch.__version__ + " (MIOpen convolutions)",
               "layout": "channels_last", "dtype": wl.dtype,
               "eager_ms_per_step": eager_s * 1e3 / steps,
               "eager_images_per_s": wl.batch * steps / eager_s}
        try:
            s = torch.cuda.Stream()
            s.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(s):
                for _ in range(3):
                    fwd(x)
            torch.cuda.current_stream().wait_stream(s)
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                y_graph = fwd(x)
            for _ in range(warmup):
                g.replay()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for _ in range(steps):
                g.replay()
            torch.cuda.synchronize()
            graph_s = time.perf_counter() - t0
            res["graph_ms_per_step"] = graph_s * 1e3 / steps
            res["graph_images_per_s"] = wl.batch * steps / graph_s
            res["graph_equals_eager"] = bool(torch.equal(y_graph, y_eager))
        except Exception as e:  # capture is best effort: report eager only
            res["graph_error"] = f"{type(e).__name__}: {e}"[:200]
    if ref_out is not None:
        yr = y_eager.float()
        if yr.dim() == 4:
            yr = yr.permute(0, 2, 3, 1)
        yr = yr.reshape(ref_out.shape)
        d = (yr - ref_out.float()).abs().max().item()
        res["max_abs_diff_vs_path"] = d
        res["max_rel_diff_vs_path"] = d / max(ref_out.float().abs().max().item(), 1e-30)
    return res


def parse_batches(spec):
    if "-" in spec and "," not in spec:
        lo, hi = (int(v) for v in spec.split("-"))
        return list(range(lo, hi + 1))
    return [int(v) for v in spec.split(",")]


def latency_table(args):
    """Per-layer latency table L[i][b] (microseconds, median over runs of the
    range in layer order, events recorded by each layer's first and last
    launch) of the workload's partition, with the feature-map size S_i,
    each layer's algorithmic work and roofline position, and the measured
    whole-partition latency next to the sum of its layers (the paper's
    planner assumes partition latency = sum of layer latencies)."""
    import numpy as np
    import torch
    import workloads as W
    from paper_2507_18748_amd import Partition
    wl = W.workload(args.workload)
    batches = parse_batches(args.batches)
    m = wl.build_model()
    P = wl.params(m)
    torch.cuda.set_device(0)
    part = Partition(m.layers, P, (m.in_c, m.in_h, m.in_w), wl.begin, wl.end, wl.dtype,
                     max_batch=max(batches))
    peak_f = PEAK_MFMA_TFLOPS[wl.dtype] * 1e12
    peak_b = PEAK_HBM_GBS * 1e9
    rows = []
    table = np.zeros((wl.end - wl.begin, len(batches)))
    whole = np.zeros(len(batches))
    chunk = 8
    for c0 in range(0, len(batches), chunk):
        bs = batches[c0:c0 + chunk]
        t, w = part.profile_layers(bs, warmup=args.profile_warmup, reps=args.profile_reps)
        table[:, c0:c0 + len(bs)] = t
        whole[c0:c0 + len(bs)] = w
        print(f"[table] batches {bs[0]}..{bs[-1]} done", file=sys.stderr, flush=True)
    for i in range(wl.begin, wl.end):
        info = part.layer_info(i, batches[-1])
        row = {"layer": i, "name": m.layers[i].name, "op": m.layers[i].op,
               "S_i_bytes": info["out_bytes_b1"], "out_chw": [info["out_c"], info["out_h"], info["out_w"]],
               "us": [], "roofline_frac": [], "bound": []}
        for j, b in enumerate(batches):
            li = part.layer_info(i, b)
            fl = b * li["flops_b1"]
            by = b * li["act_bytes_b1"] + li["param_bytes"]
            t_roof = max(fl / peak_f, by / peak_b)
            us = float(table[i - wl.begin, j])
            row["us"].append(us)
            row["roofline_frac"].append(t_roof * 1e6 / us if us > 0 else None)
            row["bound"].append("mfma" if fl / peak_f >= by / peak_b else "hbm")
        row["kernel_at_max_batch"] = info["kernel"]
        rows.append(row)
    out = {"workload": wl.name, "description": wl.description, "dtype": wl.dtype,
           "layers": [wl.begin, wl.end], "batches": batches,
           "partition_us": [float(v) for v in whole],
           "sum_of_layers_us": [float(v) for v in table.sum(axis=0)],
           "images_per_s": [b / (whole[j] * 1e-6) for j, b in enumerate(batches)],
           "method": f"layers: median of {args.profile_reps} runs (after {args.profile_warmup} "
                     "warm-up runs) of the range in layer order, HIP events recorded by each "
                     "layer's first and last kernel launch; partition: one captured HIP graph "
                     "replayed back to back",
           "rows": rows}
    write_table_json(args.table, out)
    print(json.dumps({"table": args.table, "workload": wl.name, "batches": len(batches),
                      "partition_us": dict(zip(batches, out["partition_us"]))}))
    part.close()


def blocks_report(args):
    """Pre-partitioning (Sec. 5.2) on the measured table: the workload's range
    is grouped into about N blocks of equal latency at the planning batch,
    each block is then profiled as a partition of its own at every batch (the
    block-latency table the planner consumes), and two additivity checks are
    reported: the sum of a block's layer latencies against the block measured
    alone, and the sum of the blocks against the whole range measured."""
    import numpy as np
    import torch
    import workloads as W
    from paper_2507_18748_amd import Partition, split_points, prepartition
    wl = W.workload(args.workload)
    batches = parse_batches(args.batches)
    plan_b = wl.batch if wl.batch in batches else batches[-1]
    m = wl.build_model()
    P = wl.params(m)
    torch.cuda.set_device(0)
    in_chw = (m.in_c, m.in_h, m.in_w)
    with Partition(m.layers, P, in_chw, wl.begin, wl.end, wl.dtype,
                   max_batch=max(batches)) as part:
        table, whole = part.profile_layers(batches, warmup=args.profile_warmup, reps=args.profile_reps)
    print("[blocks] layer table done", file=sys.stderr, flush=True)
    ok = split_points(m.layers)
    local_ok = [1] + [ok[p] for p in range(wl.begin + 1, wl.end)] + [1]
    jb = batches.index(plan_b)
    bounds = [wl.begin + b for b in prepartition(
        [float(v) for v in table[:, jb]], local_ok, args.blocks)]
    blocks = []
    for bb, be in zip(bounds, bounds[1:]):
        with Partition(m.layers, P, in_chw, bb, be, wl.dtype, max_batch=max(batches)) as bp:
            bt, bw = bp.profile_layers(batches, warmup=args.profile_warmup, reps=args.profile_reps)
        layer_sum = table[bb - wl.begin:be - wl.begin].sum(axis=0)
        blocks.append({"layers": [bb, be],
                       "block_us": {b: float(bw[j]) for j, b in enumerate(batches)},
                       "sum_of_layers_us": {b: float(layer_sum[j]) for j, b in enumerate(batches)},
                       "layers_over_block": {b: float(layer_sum[j] / bw[j])
                                             for j, b in enumerate(batches)}})
        print(f"[blocks] block [{bb},{be}) done", file=sys.stderr, flush=True)
    sum_blocks = {b: sum(k["block_us"][b] for k in blocks) for b in batches}
    target = float(table[:, jb].sum()) / args.blocks
    out = {"workload": wl.name, "layers": [wl.begin, wl.end], "batches": batches,
           "n_blocks_requested": args.blocks, "planning_batch": plan_b,
           "target_block_us": target, "boundaries": bounds,
           "block_us_at_planning_batch": [k["sum_of_layers_us"][plan_b] for k in blocks],
           "whole_us": {b: float(whole[j]) for j, b in enumerate(batches)},
           "sum_of_blocks_us": sum_blocks,
           "blocks_over_whole": {b: sum_blocks[b] / float(whole[j])
                                 for j, b in enumerate(batches)},
           "blocks": blocks,
           "method": "layer table in sequence (events recorded by each layer's first and "
                     "last launch); blocks and the whole range as captured HIP graphs "
                     "replayed back to back"}
    with open(args.blocks_out, "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps({"blocks": args.blocks_out, "boundaries": bounds,
                      "blocks_over_whole": out["blocks_over_whole"]}))


def serving_plan(table, out_bytes, bounds, batches, n_nodes=12, per_node=8, bs=8,
                 link_gbps=400.0, link_fixed_us=5.0):
    """A pooled-pipeline plan over a measured layer table for the request
    scheduler: three pipelines sharing n_nodes x per_node GPUs, cut at
    pre-partitioning block boundaries, pools sized to their stage's latency
    at the unified batch size `bs`.
      P0: two stages cut at the boundary nearest half the model's latency,
      P1: three stages cut nearest the thirds,
      P2: the whole model on one pool (no partitioning).
    Stage latency at batch b is the sum of its layers' latencies (partition
    latency adds up, Sec. 5.1); the transfer into a stage moves the previous
    layer's output, out_bytes[j - 1] * b bytes, over a node link of
    link_gbps plus a fixed link_fixed_us."""
    import numpy as np
    n_gpus = n_nodes * per_node
    jb = batches.index(bs)
    cum = np.concatenate([[0.0], np.cumsum(table[:, jb])])
    total = cum[-1]

    def cut(frac):
        return min(bounds[1:-1], key=lambda b: abs(cum[b] - frac * total))

    shapes = [[0, cut(0.5), len(table)],
              [0, cut(1 / 3), cut(2 / 3), len(table)],
              [0, len(table)]]
    shares = [32, 36, 28]
    gpu_node = [g // per_node for g in range(n_gpus)]
    nxt, pipes = 0, []
    for sh, share in zip(shapes, shares):
        lat = [float(cum[e] - cum[b]) for b, e in zip(sh, sh[1:])]
        pools = [max(1, int(round(share * v / sum(lat)))) for v in lat]
        pools[-1] = share - sum(pools[:-1])
        stages = []
        for (b, e), k in zip(zip(sh, sh[1:]), pools):
            infer = [float(table[b:e, j].sum()) for j in range(len(batches))]
            moved = out_bytes[b - 1] if b > 0 else 0
            net = [link_fixed_us + moved * bb / (link_gbps / 8 * 1e3) for bb in batches]
            stages.append({"gpus": list(range(nxt, nxt + k)), "infer": infer, "net": net,
                           "layers": [b, e]})
            nxt += k
        pipes.append({"bs": bs, "stages": stages})
    return gpu_node, pipes


def batching_report(args):
    """Resource-reservation adaptive batching (Sec. 5.4) fed by the measured
    per-layer table: the layer table of the workload is measured at every
    batch 1..B, cut into pre-partitioning blocks, turned into a 96-GPU
    pooled-pipeline plan, and the native scheduler then serves seeded
    Poisson and bursty request streams at several loads.  Reports drops,
    deadline misses (must be 0), reservation overlaps (must be 0) and the
    host cost of a decision."""
    import numpy as np
    import torch
    import workloads as W
    from workloads import serving as ws
    from paper_2507_18748_amd import Partition, Batcher, split_points, prepartition
    wl = W.workload(args.workload)
    batches = parse_batches(args.batches)
    if batches != list(range(1, batches[-1] + 1)):
        raise SystemExit("--batching needs every batch 1..B (e.g. --batches 1-16)")
    m = wl.build_model()
    P = wl.params(m)
    torch.cuda.set_device(0)
    in_chw = (m.in_c, m.in_h, m.in_w)
    with Partition(m.layers, P, in_chw, wl.begin, wl.end, wl.dtype,
                   max_batch=max(batches)) as part:
        table, whole = part.profile_layers(batches, warmup=args.profile_warmup, reps=args.profile_reps)
        out_bytes = [part.layer_info(i, 1)["out_bytes_b1"] for i in range(wl.begin, wl.end)]
    print("[batching] layer table done", file=sys.stderr, flush=True)
    ok = split_points(m.layers)
    local_ok = [1] + [ok[p] for p in range(wl.begin + 1, wl.end)] + [1]
    bs = min(8, batches[-1])
    bounds = prepartition([float(v) for v in table[:, batches.index(bs)]], local_ok, args.blocks)
    gpu_node, pipes = serving_plan(table, out_bytes, bounds, batches, bs=bs)
    cap = ws.plan_capacity_per_us(pipes)
    path_us = max(sum(s["infer"][bs - 1] + s["net"][bs - 1] for s in p["stages"]) for p in pipes)
    slo = 2.0 * path_us
    runs = []
    for kind in ("poisson", "bursty"):
        for load in (0.5, 0.8, 0.95):
            gen = ws.poisson_arrivals if kind == "poisson" else ws.bursty_arrivals
            arr = gen(cap * load, args.requests, 17)
            with Batcher(gpu_node, pipes) as b:
                st, _ = b.simulate(arr, slo)
                overlaps, held = b.check()
            nb = max(st["batches"], 1)
            runs.append({"arrivals": kind, "load": load, "requests": st["requests"],
                         "dropped_frac": st["dropped"] / st["requests"], "late": st["late"],
                         "overlaps": overlaps, "reservations": held,
                         "mean_batch": st["dispatched"] / nb,
                         "dispatch_probes": st["dispatch_probes"] / nb,
                         "dispatch_us": st["dispatch_us"] / nb,
                         "probes_per_batch_all": st["probes"] / nb,
                         "us_per_batch_all": st["decision_us"] / nb,
                         "served_per_s": st["dispatched"] / (arr[-1] * 1e-6)})
            print(f"[batching] {kind} load {load}: {runs[-1]}", file=sys.stderr, flush=True)
    plan = [{"bs": p["bs"], "stages": [{"layers": s["layers"], "gpus": len(s["gpus"]),
                                        f"infer_us_b{bs}": s["infer"][bs - 1],
                                        f"net_us_b{bs}": s["net"][bs - 1]} for s in p["stages"]]}
            for p in pipes]
    out = {"workload": wl.name, "batches": batches, "blocks": [wl.begin + b for b in bounds],
           "gpus": len(gpu_node), "nodes": max(gpu_node) + 1, "plan": plan,
           "capacity_per_s": cap * 1e6, "slo_us": slo, "runs": runs,
           "arrivals": "seeded synthetic (Poisson; bursty = Poisson bursts of geometric size)"}
    with open(args.batching_out, "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps({"batching": args.batching_out, "slo_us": slo,
                      "capacity_per_s": out["capacity_per_s"],
                      "runs": [{k: r[k] for k in ("arrivals", "load", "dropped_frac", "late",
                                                  "overlaps", "dispatch_probes", "dispatch_us")}
                               for r in runs]}))


def vgpu_report(args):
    """Latency under virtual GPUs (Sec. 5.3): for k = 1..4 the GPU's compute
    units are split into k equal shares (CU-masked streams; the paper uses
    MPS) and the same partition runs on every share side by side, one handle
    per share, each replaying its captured graph, so the interference
    between co-located shares is part of the measurement (the paper profiles
    the same way).  Reports per batch each share's latency and the GPU's
    aggregate images/s."""
    import numpy as np
    import torch
    import workloads as W
    from paper_2507_18748_amd import Partition, stream_cu_share, stream_destroy
    wl = W.workload(args.workload)
    batches = parse_batches(args.batches)
    m = wl.build_model()
    P = wl.params(m)
    torch.cuda.set_device(0)
    tdt = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}[wl.dtype]
    x = wl.input(max(batches))
    xh = torch.from_numpy(np.ascontiguousarray(x.transpose(0, 2, 3, 1))).to(tdt)
    reps = args.vgpu_reps
    out = {"workload": wl.name, "layers": [wl.begin, wl.end], "batches": batches,
           "shares": {}, "method": "k handles on k CU-masked streams (CU i in share (i/8) mod k), "
                                   "graphs replayed side by side; latency = elapsed / reps per "
                                   "stream, HIP events on each stream; each handle planned for "
                                   + ("the whole device" if args.vgpu_whole_plans else
                                      "its share's CUs (ppipe_partition_create_on_share)")}
    for k in (1, 2, 3, 4):
        parts = [Partition(m.layers, P, (m.in_c, m.in_h, m.in_w), wl.begin, wl.end, wl.dtype,
                           max_batch=max(batches),
                           cu_share_parts=None if args.vgpu_whole_plans else k)
                 for _ in range(k)]
        streams = [stream_cu_share(j, k) for j in range(k)]
        ext = [torch.cuda.ExternalStream(st) for st in streams]
        info = parts[0].info
        odt = torch.float32 if info["out_dtype"] == 0 else tdt
        ins = [xh.cuda() for _ in range(k)]
        outs = [torch.empty((max(batches), info["out_h"], info["out_w"], info["out_c"]),
                            dtype=odt, device="cuda") for _ in range(k)]
        rows = {}
        for b in batches:
            for j in range(k):
                parts[j].capture(b, ins[j].data_ptr(), outs[j].data_ptr())
            for _ in range(3):
                for j in range(k):
                    parts[j].run(b, ins[j].data_ptr(), outs[j].data_ptr(), streams[j])
            torch.cuda.synchronize()
            e0 = [torch.cuda.Event(enable_timing=True) for _ in range(k)]
            e1 = [torch.cuda.Event(enable_timing=True) for _ in range(k)]
            for j in range(k):
                e0[j].record(ext[j])
            for _ in range(reps):
                for j in range(k):
                    parts[j].run(b, ins[j].data_ptr(), outs[j].data_ptr(), streams[j])
            for j in range(k):
                e1[j].record(ext[j])
            torch.cuda.synchronize()
            lat = [e0[j].elapsed_time(e1[j]) * 1e3 / reps for j in range(k)]
            rows[b] = {"latency_us": lat, "mean_latency_us": float(np.mean(lat)),
                       "images_per_s": float(sum(b / (t * 1e-6) for t in lat))}
        out["shares"][k] = rows
        print(f"[vgpu] {k} share(s) done: b={batches[-1]} mean "
              f"{rows[batches[-1]]['mean_latency_us']:.1f} us", file=sys.stderr, flush=True)
        torch.cuda.synchronize()
        for p_ in parts:
            p_.close()
        for st in streams:
            stream_destroy(st)
    with open(args.vgpu_out, "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps({"vgpu": args.vgpu_out, "workload": wl.name,
                      "images_per_s_at_max_batch": {k: v[batches[-1]]["images_per_s"]
                                                    for k, v in out["shares"].items()}}))


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2000)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--batch", type=int, default=0,
                    help="batch of the benchmark (default: 64 for resnet152, else the "
                         "workload's own batch)")
    ap.add_argument("--no-graph", action="store_true", help="launch kernels directly")
    ap.add_argument("--blocks-out", default="", metavar="OUT.json",
                    help="pre-partition the workload into --blocks blocks from its latency "
                         "table and write block tables and additivity checks")
    ap.add_argument("--blocks", type=int, default=10, help="N of the pre-partitioning")
    ap.add_argument("--vgpu-out", default="", metavar="OUT.json",
                    help="latency of the workload on 1/1, 1/2, 1/3, 1/4 CU shares run side by side")
    ap.add_argument("--vgpu-reps", type=int, default=20)
    ap.add_argument("--batching-out", default="", metavar="OUT.json",
                    help="serve synthetic request streams with the adaptive batching "
                         "scheduler over the workload's measured table (--batches 1-B)")
    ap.add_argument("--requests", type=int, default=200000)
    ap.add_argument("--vgpu-whole-plans", action="store_true",
                    help="with --vgpu-out: plan every share's handle for the whole device "
                         "(the default plans each for its share's CUs)")
    ap.add_argument("--sweep-batches", default="1,2,4,8,16,32,64", metavar="LIST",
                    help="also time graph replays of the same handle at these batches "
                         "(up to the workload's batch) and report images/s per batch; 'none' "
                         "skips")
    ap.add_argument("--cold-reps", type=int, default=5,
                    help="isolated-cold repetitions per launch (caches swept before each); "
                         "0 skips")
    ap.add_argument("--timing-steps", type=int, default=20,
                    help="directly launched steps whose per-launch events give the roofline")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="oracle sample length for cpu_baseline (0 disables)")
    ap.add_argument("--profile-reps", type=int, default=50,
                    help="timed repetitions per latency-table entry (median)")
    ap.add_argument("--profile-warmup", type=int, default=10,
                    help="untimed repetitions before the latency-table runs")
    ap.add_argument("--table", metavar="OUT.json", default=None,
                    help="instead of the benchmark, write the per-layer latency table of the "
                         "workload (median us per layer at each --batches size) with S_i and "
                         "per-layer roofline fractions")
    ap.add_argument("--batches", default="1-64",
                    help="batch sizes for --table: '1-64', or a comma list")
    ap.add_argument("--kernels", metavar="OUT.json", default=None,
                    help="also write every launch's timing record of the benchmark batch")
    ap.add_argument("--library-baseline", action="store_true",
                    help="also time the same partition on PyTorch-ROCm's own kernels "
                         "(MIOpen convolutions) and add it to the line as library_baseline")
    ap.add_argument("--traffic-record", metavar="OUT.json", default=None,
                    help="write the dominant kernel's HBM-traffic record from rocprofv3 --pmc "
                         "csv directories under --pmc-dir (needs --traffic-from)")
    ap.add_argument("--traffic-from", metavar="BENCH.json", default=None,
                    help="bench.py output line naming the dominant kernel")
    ap.add_argument("--pmc-dir", default="gpurun_out/pmc")
    ap.add_argument("--pmc-commands", default="", help="';'-separated commands that made the csvs")
    ap.add_argument("--copy-mib", type=float, default=256.0)
    ap.add_argument("--launch-floor", action="store_true",
                    help="only time graphs of 200 back-to-back dependent launches of tiny "
                         "kernels (the per-launch floor under a partition) and exit")
    ap.add_argument("--copy-calibration", type=float, default=0.0, metavar="MIB",
                    help="only run a plain device-to-device copy of MIB mebibytes 10 times "
                         "(reference for the HBM byte counters) and exit")
    args = ap.parse_args()

    if args.traffic_record:
        return traffic_record(args)
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on one GPU only: the partition forward is measured on a single "
              "MI355X (data parallelism over more GPUs needs no exchange and is not "
              "launched here)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    if args.copy_calibration > 0:
        n = int(args.copy_calibration * 2 ** 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(10):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": n * 4, "repeats": 10}))
        return
    if args.launch_floor:
        print(json.dumps(launch_floor()))
        return
    import workloads as W
    from paper_2507_18748_amd import Partition

    if args.table:
        return latency_table(args)
    if args.blocks_out:
        return blocks_report(args)
    if args.vgpu_out:
        return vgpu_report(args)
    if args.batching_out:
        return batching_report(args)

    wl = W.workload(args.workload)
    batch = args.batch or DEFAULT_BATCH.get(wl.name, wl.batch)
    if batch != wl.batch:
        import dataclasses
        wl = dataclasses.replace(wl, batch=batch)
    m = wl.build_model()
    P = wl.params(m)
    torch.cuda.set_device(0)
    part = Partition(m.layers, P, (m.in_c, m.in_h, m.in_w), wl.begin, wl.end, wl.dtype,
                     max_batch=wl.batch)
    tdt = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}[wl.dtype]
    x = wl.input(wl.batch)
    xd = torch.from_numpy(np.ascontiguousarray(x.transpose(0, 2, 3, 1))).to(tdt).cuda()
    info = part.info
    odt = torch.float32 if info["out_dtype"] == 0 else tdt
    out = torch.empty((wl.batch, info["out_h"], info["out_w"], info["out_c"]), dtype=odt,
                      device="cuda")
    stream = torch.cuda.current_stream()
    sp = stream.cuda_stream
    if not args.no_graph:
        part.capture(wl.batch, xd.data_ptr(), out.data_ptr())
    for _ in range(args.warmup):
        part.run(wl.batch, xd.data_ptr(), out.data_ptr(), sp)
    torch.cuda.synchronize()
    print(f"[bench] {wl.name} batch {wl.batch}: warmup done", file=sys.stderr, flush=True)

    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        part.run(wl.batch, xd.data_ptr(), out.data_ptr(), sp)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_ms = ev0.elapsed_time(ev1)
    assert torch.isfinite(out.float()).all()
    print(f"[bench] timed {args.steps} steps: wall {wall * 1e3:.2f} ms, events {gpu_ms:.2f} ms",
          file=sys.stderr, flush=True)

    # Launch durations: right after the timed region, steps launched directly
    # in the same layer order, each launch recording a pair of HIP events
    # around the kernel itself on the stream the kernels run on (events inside
    # a replayed graph cannot be timed on ROCm).  Mean over the steps.
    part.timing_setup(wl.batch, xd.data_ptr(), out.data_ptr())
    part.run_timed(sp)
    recs = None
    for _ in range(args.timing_steps):
        part.run_timed(sp)
        r = part.timing_read()
        if recs is None:
            recs = r
        else:
            for a, b in zip(recs, r):
                a["mean_us"] += b["mean_us"]
    for a in recs:
        a["mean_us"] /= args.timing_steps
        a["median_us"] = a["min_us"] = a["mean_us"]
    roof = roofline(recs, wl.dtype)
    roof["traffic"] = measured_traffic(wl.name, roof["kernel"], wl.batch)
    roof["timing"] = (f"HIP events recorded by each launch, {args.timing_steps} directly "
                      f"launched steps after the timed region")
    if args.kernels:
        with open(args.kernels, "w") as f:
            json.dump(recs, f, indent=1)
    print(f"[bench] dominant kernel {roof['kernel']}: {roof['achieved']:.1f} {roof['unit']} "
          f"({roof['frac'] * 100:.1f}% of peak)", file=sys.stderr, flush=True)

    result = {
        "metric": METRIC,
        "value": wl.batch * args.steps / wall,
        "unit": "images/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": wall * 1e3 / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": DTYPE_LABEL[wl.dtype],
        "data": "synthetic (seeded He-init weights, seeded inputs; no trained weights)",
        "config": {"workload": wl.description, "name": wl.name, "layers": [wl.begin, wl.end],
                   "batch": wl.batch, "input": "x".join(map(str, (wl.batch,) + wl.in_chw)) +
                   f" {wl.dtype} {wl.input_kind}", "graph": not args.no_graph},
        "roofline": roof,
    }
    if args.cold_reps > 0:
        cold = part.profile_kernels_cold(wl.batch, reps=args.cold_reps)
        cref = copy_reference()
        result["isolated_cold"] = cold_summary(cold, wl.dtype, cref["cold_fit"])
        result["isolated_cold"]["copy_reference"] = cref
    if args.sweep_batches and args.sweep_batches != "none":
        result["batch_sweep"] = batch_sweep(part, wl.batch, xd, out, sp,
                                            parse_batches(args.sweep_batches))
    if args.library_baseline:
        print("[bench] timing the PyTorch-ROCm library baseline", file=sys.stderr, flush=True)
        part.run(wl.batch, xd.data_ptr(), out.data_ptr(), sp)
        torch.cuda.synchronize()
        lb = library_baseline(wl, m, P, x, min(args.steps, 500), 20, out)
        lb["path_over_library_graph"] = (lb["graph_ms_per_step"] / result["ms_per_step"]
                                         if "graph_ms_per_step" in lb else None)
        result["library_baseline"] = lb
    if args.cpu_seconds > 0:
        print("[bench] timing the CPU oracle", file=sys.stderr, flush=True)
        result["cpu_baseline"] = cpu_baseline(wl, m, P, args.cpu_seconds)
    part.close()
    print(json.dumps(result))


if __name__ == "__main__":
    main()

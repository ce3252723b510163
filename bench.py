"""Benchmark: one GPU's share of a training step of the encoder-decoder.

A step is one pass of the whole hot path over one synthetic batch: the
forward pass of the 13 layers (fused ReLU), the loss-scaled L2 head
gradient, the backward pass (kernel and input gradients, fused ReLU
gradient) and, as each group of weight gradients completes, fusion-buffer
pack, unscale with overflow check and unpack into fp32 master gradients
(25 MiB groups). Inputs are resident in HBM before the timed region.

value = algorithmic convolution flops of the step (3 passes x 13 layers,
direct-convolution count, 5.528 TFLOP) / wall time of the step, in TFLOP/s.
The JSON line also carries the roofline of the dominant kernel (timed with
HIP events on its own stream inside the timed region), the gradient-path
bandwidths and the CPU oracle timed on a bounded sample of the same work.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu]
       python bench.py --op E2b.fwd|E2b.dx|E2b.dW|copy [--steps K]
       python bench.py --summarize-stats CSV
       python bench.py --summarize-pmc DIR
The --op form runs one pass of one layer (seeded full-size inputs) K times
and prints its per-launch time; `copy` is a plain 256 MiB fp16 copy through
grad_group_pack, the reference for scaling HBM byte counters.
--summarize-stats turns a rocprofv3 --stats kernel_stats.csv into a markdown
table; --summarize-pmc turns four rocprofv3 --pmc runs (DIR/step_FETCH_SIZE,
DIR/step_WRITE_SIZE, DIR/copy_FETCH_SIZE, DIR/copy_WRITE_SIZE, each holding
run_counter_collection.csv) into a per-kernel HBM traffic table plus the
machine-readable lines recorded_traffic() reads.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

MFMA_F16_PEAK_TFLOPS = 2500.0      # MI355X dense fp16 MFMA
HBM_PEAK_GBPS = 8000.0             # MI355X HBM3E


def paper_rates(ops_conv_per_pass, t_exec_s, t_comp_s):
    """Sustained and Peak performance of Section 5.2 (flop/s): the three
    convolution passes of a step (forward, kernel gradient, input gradient),
    3 * OPS_conv, over the step's execution time t_exec and over the time its
    convolutions compute, t_comp."""
    total = 3.0 * ops_conv_per_pass
    return total / t_exec_s, total / t_comp_s


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--settle-steps", type=int, default=200,
                    help="untimed steps of the timed program run back to back before the "
                         "warm-up steps (the first steps after the one-stream detail pass "
                         "run 1-1.4%% slower than the steady state)")
    ap.add_argument("--no-cpu", action="store_true",
                    help="skip the CPU oracle baseline leg")
    ap.add_argument("--cpu-seconds", type=float, default=20.0,
                    help="approximate CPU work of the oracle sample")
    ap.add_argument("--detail", default=None,
                    help="write per-op timings (JSON) to this path")
    ap.add_argument("--streams", type=int, default=3, choices=(1, 3),
                    help="streams of the timed step (3: kernel gradients and the "
                         "gradient path beside the input-gradient chain)")
    ap.add_argument("--zero-copy", action="store_true",
                    help="kernel gradients write into their group slots (no pack; "
                         "the non-finite check fused into their store)")
    ap.add_argument("--workload", default="fcn", choices=("fcn", "densenet"),
                    help="fcn: the encoder-decoder step; densenet: the FC-DenseNet "
                         "variant's step (25 MiB gradient groups; with --streams 3 its kernel "
                         "gradients and the gradient path run on a second stream)")
    ap.add_argument("--optimizer", action="store_true",
                    help="end each step with the layer-wise adaptive Adam update of "
                         "fp32 master weights under a backoff loss scale")
    ap.add_argument("--op", default=None,
                    help="time one pass of one layer, e.g. E2b.fwd, or 'copy'")
    ap.add_argument("--summarize-stats", default=None, metavar="CSV")
    ap.add_argument("--summarize-pmc", default=None, metavar="DIR")
    ap.add_argument("--summarize-trace", nargs=2, default=None, metavar=("CSV", "KERNEL"),
                    help="durations of KERNEL in a kernel trace of a bench run (pass the "
                         "traced run's --steps, --warmup and the kernel's "
                         "--launches-per-step)")
    ap.add_argument("--launches-per-step", type=int, default=6,
                    help="with --summarize-trace: the kernel's launches per step")
    ap.add_argument("--summarize-mfma", default=None, metavar="DIR",
                    help="per-kernel MFMA utilisation table from two rocprofv3 --pmc "
                         "runs (DIR/mfma_busy, DIR/mfma_ops)")
    ap.add_argument("--grad-path-only", action="store_true",
                    help="only the standalone, cache-flushed gradient-path measurement")
    ap.add_argument("--grad-reps", type=int, default=20,
                    help="reps per group and kernel of the gradient-path measurement")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the standalone gradient path and the small configurations")
    ap.add_argument("--ceiling", action="store_true",
                    help="measure the practical MFMA ceiling instead: clocks and power "
                         "under the sustained step and under a vendor-library GEMM, and "
                         "every pass against the vendor GEMM of the same shape")
    ap.add_argument("--summarize-ceiling", default=None, metavar="JSON",
                    help="turn the --ceiling JSON line into markdown tables")
    ap.add_argument("--no-clocks", action="store_true",
                    help="do not query amd-smi / rocm-smi for the clocks")
    return ap.parse_args()


WORKLOADS = {
    "fcn": "fcn encoder-decoder step, N=4 x 256x256 x 256ch input, 13 layers "
           "(99,483,904 weights), L2 head, loss scale 2^15, 25 MiB gradient groups (9)",
    "densenet": "FC-DenseNet variant step, N=4 x 128x128 x 256ch input, growth 256, "
                "2 levels of 2-layer dense blocks + bottleneck, average pooling, "
                "16 conv layers (38,928,896 weights), Huber head (delta 10), "
                "loss scale 2^15, layers write into their concatenation slices and add their "
                "input gradients in place, 25 MiB gradient groups (4), kernel gradients and "
                "the gradient path on a second stream",
}

COPY_KIB = 256 * 1024  # bytes read (and written) by `--op copy`, in KiB


def short_kernel_name(name):
    """rocprofv3 kernel name -> the name fg.kernel_name() reports."""
    import re
    name = name.replace("(anonymous namespace)::", "")
    name = name.split("(")[0].replace("void ", "")
    name = name.replace("fg::dma::", "").replace("fg::", "")
    # the pipeline configuration: dropped, except a tile size other than 256
    name = re.sub(r"K<\d+, \d+, \d+, \d+(, 256)?>, ", "", name)
    return re.sub(r"K<\d+, \d+, \d+, \d+, (\d+)>, ", r"\1, ", name)


def kernel_source(kernel):
    """Source file (under paper_1909_11150_amd/csrc) that defines `kernel`."""
    if "_dma_kernel" in kernel or "_halo_kernel" in kernel:
        return "conv_dma.hip"
    if kernel.startswith(("copy_pieces", "unscale", "head_grad", "relu_backward")):
        return "grad_path.hip"
    return "conv_igemm.hip"


def source_hash(kernel):
    """Hash of the source file that defines `kernel` and of the one that
    holds the tile and split planner (which decides the layers and splits a
    kernel runs, and so its bytes per launch)."""
    import hashlib
    h = hashlib.sha256()
    for f in dict.fromkeys((kernel_source(kernel), "conv_igemm.hip")):
        h.update(open(os.path.join(ROOT, "paper_1909_11150_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def summarize_stats(path):
    import csv
    print("| kernel | calls | total ms | avg us | % | min us | max us |")
    print("|---|---:|---:|---:|---:|---:|---:|")
    for r in csv.DictReader(open(path)):
        print(f"| `{short_kernel_name(r['Name'])}` | {r['Calls']} | "
              f"{float(r['TotalDurationNs']) / 1e6:.3f} | {float(r['AverageNs']) / 1e3:.2f} | "
              f"{float(r['Percentage']):.2f} | {float(r['MinNs']) / 1e3:.2f} | "
              f"{float(r['MaxNs']) / 1e3:.2f} |")


def summarize_trace(path, kernel, per_step, timed_steps, warmup, settle):
    """Launch durations of one kernel from a rocprofv3 kernel trace of the
    default bench command. The step program runs warmup + 4 one-stream steps
    (warm-up, two detail steps timing calls, two timing main kernels), then
    settle + warmup + timed_steps steps on the timed streams; launches
    of the kernel by the measurements that follow (single steps, the clock
    sampling, gradient path, small configurations) come after those and are
    left out."""
    import csv
    rows = [r for r in csv.DictReader(open(path))
            if short_kernel_name(r["Kernel_Name"]) == kernel]
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    dur = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 for r in rows]
    one = warmup + 4
    total = one + settle + warmup + timed_steps
    step_dur = dur[:per_step * total]
    timed = step_dur[-per_step * timed_steps:]
    alone = step_dur[per_step * warmup:per_step * one]
    print(f"`{kernel}`: {len(step_dur)} launches in the {total} steps, average "
          f"{sum(step_dur) / len(step_dur):.2f} us; one-stream detail steps: {len(alone)} "
          f"launches, average {sum(alone) / len(alone):.2f} us; timed region (last "
          f"{timed_steps} steps): {len(timed)} launches, average "
          f"{sum(timed) / len(timed):.2f} us")


def summarize_pmc(d):
    import csv

    def per_kernel(run):
        out = {}
        for r in csv.DictReader(open(os.path.join(d, run, "run_counter_collection.csv"))):
            k = short_kernel_name(r["Kernel_Name"])
            v = out.setdefault(k, [0, 0.0])
            v[0] += 1
            v[1] += float(r["Counter_Value"])
        return {k: (n, tot / n) for k, (n, tot) in out.items()}

    cf, cw = per_kernel("copy_FETCH_SIZE"), per_kernel("copy_WRITE_SIZE")
    cname = "copy_pieces_kernel<2>"
    fscale = COPY_KIB / cf[cname][1]
    wscale = COPY_KIB / cw[cname][1]
    print(f"Calibration: a plain copy of {COPY_KIB} KiB (read, and the same written) "
          f"reads FETCH_SIZE {cf[cname][1]:.0f} KiB and WRITE_SIZE {cw[cname][1]:.0f} KiB "
          f"per dispatch, so the scale factors are fetch x{fscale:.3f}, write x{wscale:.3f}.")
    print()
    sf, sw = per_kernel("step_FETCH_SIZE"), per_kernel("step_WRITE_SIZE")
    rows = []
    for k in sf:
        if k not in sw:
            continue
        mb = (sf[k][1] * fscale + sw[k][1] * wscale) * 1024 / 1e6
        rows.append((mb * sf[k][0], k, sf[k][0], sf[k][1], sw[k][1], mb))
    rows.sort(reverse=True)
    print("| kernel | dispatches | FETCH_SIZE KiB per dispatch (raw) | "
          "WRITE_SIZE KiB per dispatch (raw) | scaled MB per dispatch |")
    print("|---|---:|---:|---:|---:|")
    for _, k, n, f, w, mb in rows[:16]:
        print(f"| `{k}` | {n} | {f:.0f} | {w:.0f} | {mb:.1f} |")
    print()
    print("Machine-readable lines for bench.py (kernel, hash of the source file "
          "that defines it when measured, scaled HBM bytes per dispatch averaged "
          "over the kernel's dispatches in the step):")
    print()
    for _, k, n, f, w, mb in rows:
        if k.startswith(("data_conv", "wgrad")):
            print(f"traffic: kernel={k} src_sha256_16={source_hash(k)} "
                  f"bytes_per_launch={int(round(mb * 1e6))}")
    if os.path.isdir(os.path.join(d, "gp_FETCH_SIZE")):
        # the standalone gradient path (--grad-path-only): per dispatch of
        # each kernel, against its algorithmic bytes
        # each thread of the three kernels moves 16 elements (the grid is
        # rounded up to whole workgroups, so this is an upper bound)
        bpe = {"copy_pieces_kernel<2>": 4, "unscale_vec_kernel": 6, "copy_pieces_kernel<4>": 8}

        def algo_and_counted(run):
            out = {}
            for r in csv.DictReader(open(os.path.join(d, run, "run_counter_collection.csv"))):
                k = short_kernel_name(r["Kernel_Name"])
                if k in bpe:
                    v = out.setdefault(k, [0, 0.0, 0.0])
                    v[0] += 1
                    v[1] += float(r["Counter_Value"])
                    v[2] += int(r["Grid_Size"]) * 16 * bpe[k]
            return out
        gf, gw = algo_and_counted("gp_FETCH_SIZE"), algo_and_counted("gp_WRITE_SIZE")
        print()
        print("Standalone gradient path (`--grad-path-only`: the nine groups, each alone and "
              "back to back, and single launches of 4 to 256 MiB), caches evicted before "
              "each launch:")
        print()
        print("| kernel | dispatches | counted MB (scaled), all dispatches | algorithmic MB, "
              "all dispatches | ratio |")
        print("|---|---:|---:|---:|---:|")
        for k in bpe:
            if k in gf and k in gw:
                mb = (gf[k][1] * fscale + gw[k][1] * wscale) * 1024 / 1e6
                algo = gf[k][2] / 1e6
                print(f"| `{k}` | {gf[k][0]} | {mb:.0f} | {algo:.0f} | {mb / algo:.3f} |")


def summarize_mfma(d):
    """Per-kernel MFMA utilisation from one rocprofv3 --pmc run of the
    derived MfmaUtil (MFMA-busy cycles summed over the SIMDs / (GPU-active
    cycles x SIMDs), in %) with SQ_INSTS_VALU_MFMA_MOPS_F16 (x 512 = the
    flops the matrix cores executed, padding of partial tiles included),
    SQ_LDS_BANK_CONFLICT and SQ_LDS_IDX_ACTIVE (a *counter_collection.csv
    under DIR). Averages over each kernel's dispatches."""
    import csv
    import glob
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    disp = {}
    for f in files:
        for r in csv.DictReader(open(f)):
            key = (f, r["Dispatch_Id"])
            e = disp.setdefault(key, {"kernel": short_kernel_name(r["Kernel_Name"])})
            name = r["Counter_Name"]
            for suf in ("_sum", "_max", "_min", "_avr"):
                if name.endswith(suf):
                    name = name[:-len(suf)]
            e[name] = e.get(name, 0.0) + float(r["Counter_Value"])
    per = {}
    for e in disp.values():
        if "MfmaUtil" not in e:
            continue
        k = per.setdefault(e["kernel"], [0, 0.0, 0.0, 0.0, 0.0])
        k[0] += 1
        k[1] += e["MfmaUtil"]
        k[2] += e.get("SQ_INSTS_VALU_MFMA_MOPS_F16", 0.0) * 512
        k[3] += e.get("SQ_LDS_BANK_CONFLICT", 0.0)
        k[4] += e.get("SQ_LDS_IDX_ACTIVE", 0.0)
    print("| kernel | dispatches | MFMA busy (MfmaUtil) | MFMA GFLOP per dispatch | "
          "LDS bank-conflict cycles / LDS-active cycles |")
    print("|---|---:|---:|---:|---:|")
    for k, (n, util, fl, bc, act) in sorted(per.items(), key=lambda kv: -kv[1][2]):
        if fl == 0:
            continue
        conf = f"{100 * bc / act:.1f}%" if act else "-"
        print(f"| `{k}` | {n} | {util / n:.1f}% | {fl / n / 1e9:.2f} | {conf} |")


def _op_call(label, rng):
    """(callable, algorithmic flops, kernel name) for one pass `LAYER.fwd|dx|dW`
    of the encoder-decoder on seeded full-size inputs."""
    import torch

    import paper_1909_11150_amd as fg
    import synth
    from paper_1909_11150_amd import fcn
    name, pas = label.split(".")
    L = {l.name: l for l in synth.fcn_layers()}[name]
    x = torch.from_numpy(np.maximum(synth.normal(rng, L.x_shape), np.float16(0))).cuda()
    w = torch.from_numpy(synth.normal(rng, L.w_shape, synth.he_std(L))).cuda()
    dy = torch.from_numpy(synth.normal(rng, L.y_shape)).cuda()
    y = torch.empty(L.y_shape, dtype=torch.float16, device="cuda")
    dx = torch.empty(L.x_shape, dtype=torch.float16, device="cuda")
    dw = torch.empty(L.w_shape, dtype=torch.float16, device="cuda")
    ws = torch.empty(max(16, fcn.chain_workspace_bytes([L])), dtype=torch.uint8,
                     device="cuda")
    d, dd = fcn.fwd_desc(L), fcn.convt_dx_desc(L)
    conv = L.kind == "conv"
    calls = {
        "fwd": (lambda: fg.conv2d_fwd(d, x, w, y, fg.EPI_RELU, None, ws),
                fg.kernel_name(d, fg.OP_FWD)) if conv else
               (lambda: fg.conv_transpose2d_fwd(d, x, w, y, fg.EPI_RELU, None, ws),
                fg.kernel_name(d, fg.OP_CONVT)),
        "dx": (lambda: fg.conv2d_bwd_data(d, dy, w, dx, fg.EPI_GATE, x, ws),
               fg.kernel_name(d, fg.OP_BWD_DATA)) if conv else
              (lambda: fg.conv2d_fwd(dd, dy, w, dx, fg.EPI_GATE, x, ws),
               fg.kernel_name(dd, fg.OP_FWD)),
        "dW": (lambda: fg.conv2d_bwd_weight(d, x, dy, dw, ws),
               fg.kernel_name(d, fg.OP_BWD_WEIGHT)) if conv else
              (lambda: fg.conv2d_bwd_weight(dd, dy, x, dw, ws),
               fg.kernel_name(dd, fg.OP_BWD_WEIGHT)),
    }
    fn, kern = calls[pas]
    return fn, L.flops, kern


def op_bench(label, steps, warmup):
    """Time one library call in isolation on seeded full-size inputs."""
    import torch

    import paper_1909_11150_amd as fg
    rng = np.random.default_rng(5)
    if label == "copy":
        n = 128 * 1024 * 1024  # 256 MiB of fp16 in, 256 MiB out
        src = torch.from_numpy(rng.integers(0, 0x7BFF, size=n, dtype=np.int16)).cuda()
        dst = torch.empty(n, dtype=torch.int16, device="cuda")
        fn = lambda: fg.grad_group_pack([src], [0], dst)
        work, unit, kern = 4 * n, "GB/s", "copy_pieces_kernel<2>"
    else:
        fn, work, kern = _op_call(label, rng)
        unit = "TFLOP/s"
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(steps)]
    for e0, e1 in evs:
        e0.record()
        fn()
        e1.record()
    torch.cuda.synchronize()
    ts = sorted(e0.elapsed_time(e1) for e0, e1 in evs)
    med = ts[len(ts) // 2] * 1e-3
    rate = work / med / (1e12 if unit == "TFLOP/s" else 1e9)
    print(json.dumps({"op": label, "kernel": kern, "median_us": round(med * 1e6, 2),
                      "min_us": round(ts[0] * 1e3, 2), "rate": round(rate, 1),
                      "unit": unit, "launches": steps}), flush=True)


def recorded_traffic(kernel, workload="fcn"):
    """HBM bytes per launch of `kernel` in the workload's step, from
    profiles/<workload>_step_hbm_traffic.md (rocprofv3 FETCH_SIZE +
    WRITE_SIZE, scaled by a plain copy's reading), or None when no record
    exists for it or the kernel's source file or the planner's has changed
    since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"{workload}_step_hbm_traffic.md")
    try:
        lines = open(path).read().splitlines()
        sha = source_hash(kernel)
    except OSError:
        return None
    for ln in lines:
        if not ln.startswith("traffic: kernel="):
            continue
        body = ln[len("traffic: kernel="):]
        name, rest = body.split(" src_sha256_16=")
        h, b = rest.split(" bytes_per_launch=")
        if name == kernel and h == sha:
            return int(b)
    return None


def cpu_baseline(layers, seconds):
    """Time the fp64 oracle on a bounded sample of the step's convolutions:
    the same seeded full-size inputs, a random sample of output elements of
    every layer's three passes, sized so the whole sample takes roughly
    `seconds`. Reported as algorithmic TFLOP/s (flops per output element x
    elements computed / time)."""
    import oracle
    threads = int(os.environ.get("OMP_NUM_THREADS", len(os.sched_getaffinity(0))))
    rng = np.random.default_rng(123)
    per_task = seconds / (3 * len(layers))
    flops_done, t_total = 0.0, 0.0
    for L in layers:
        xs = np.maximum(rng.standard_normal(L.x_shape), 0.0)
        ws = rng.standard_normal(L.w_shape)
        dys = rng.standard_normal(L.y_shape)
        ny = int(np.prod(L.y_shape))
        nx = int(np.prod(L.x_shape))
        nw = int(np.prod(L.w_shape))
        if L.kind == "conv":
            tasks = [
                (ny, lambda i: oracle.conv2d_fwd_points(xs, ws, i, L.stride, L.pad)),
                (nx, lambda i: oracle.conv2d_bwd_data_points(dys, ws, L.x_shape, i,
                                                             L.stride, L.pad)),
                (nw, lambda i: oracle.conv2d_bwd_weight_points(xs, dys, L.r, L.s, i,
                                                               L.stride, L.pad))]
        else:
            tasks = [
                (ny, lambda i: oracle.conv_transpose2d_fwd_points(xs, ws, i, 2, 1)),
                (nx, lambda i: oracle.conv2d_fwd_points(dys, ws, i, 2, 1)),
                (nw, lambda i: oracle.conv2d_bwd_weight_points(dys, xs, L.r, L.s, i,
                                                               2, 1))]
        for total, fn in tasks:
            fpe = L.flops / total   # algorithmic flops per output element
            # grow the sample until one evaluation takes half the per-task
            # budget or more (the last, largest one is the timed one)
            k = min(total, 64)
            while True:
                idx = rng.choice(total, size=k, replace=False)
                t0 = time.perf_counter()
                fn(idx)
                dt = time.perf_counter() - t0
                if k >= total or dt >= per_task / 2:
                    break
                k = min(total, k * 2)
            t_total += dt
            flops_done += fpe * k
        del xs, ws, dys
    return {"value": flops_done / t_total / 1e12, "unit": "TFLOP/s",
            "cores": threads, "kind": "oracle",
            "sample": (f"fp64 oracle on random output elements of all 39 conv "
                       f"passes of the full network (full-size seeded inputs), "
                       f"{flops_done / 1e9:.1f} GFLOP algorithmic in {t_total:.1f} s")}


def cpu_model():
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_grad_baseline(seconds):
    """The gradient path's NumPy oracle (pack, unscale with the non-finite
    check, unpack; single-threaded) on whole config-5 groups, repeated for
    about `seconds`; GB/s of the same algorithmic bytes the GPU kernels are
    credited with (4 + 6 + 8 bytes per group element)."""
    import synth
    from oracle import grad as G
    layers = synth.fcn_layers()
    numels = [L.w_numel for L in reversed(layers)]
    plan = G.plan_groups(numels, synth.GROUP_CAP_BYTES, synth.GROUP_ALIGN_BYTES)
    rng = np.random.default_rng(11)
    srcs = [synth.normal(rng, (n,), 1.0) for n in numels]
    done, t_total, groups = 0, 0.0, 0
    while t_total < seconds and groups < 64:
        g = plan[groups % len(plan)]
        t0 = time.perf_counter()
        buf = G.pack(srcs, g)
        out, _ = G.unscale_check(buf, 1.0 / synth.LOSS_SCALE)
        G.unpack(out, g, numels)
        t_total += time.perf_counter() - t0
        done += 18 * g["numel"]
        groups += 1
    return {"value": round(done / t_total / 1e9, 3), "unit": "GB/s", "cores": 1,
            "kind": "oracle",
            "sample": f"NumPy pack + unscale/check + unpack of {groups} whole gradient "
                      f"groups of the 25 MiB plan ({done / 1e9:.2f} GB algorithmic) "
                      f"in {t_total:.1f} s"}


def gpu_clocks():
    """Current clocks as amd-smi prints them: {section: first CLK value}
    for the GFX (SCLK) and MEM (MCLK) sections, or the raw clock lines of
    rocm-smi; None if neither tool answers."""
    import subprocess
    try:
        r = subprocess.run(["amd-smi", "metric", "--clock"], capture_output=True,
                           text=True, timeout=20)
        if r.returncode == 0:
            out, sec = {}, None
            for ln in r.stdout.splitlines():
                t = ln.strip()
                if t.endswith(":") and " " not in t:
                    sec = t[:-1]
                elif sec and t.startswith("CLK:") and sec not in out:
                    out[sec] = t.split(":", 1)[1].strip()
            keep = {k: v for k, v in out.items() if k.startswith(("GFX", "MEM"))}
            if keep:
                return {"tool": "amd-smi", "clk": keep}
    except (OSError, subprocess.TimeoutExpired):
        pass
    try:
        r = subprocess.run(["rocm-smi", "--showclocks"], capture_output=True, text=True,
                           timeout=20)
        if r.returncode == 0:
            return {"tool": "rocm-smi",
                    "lines": [ln.strip() for ln in r.stdout.splitlines()
                              if "clk" in ln.lower()][:8]}
    except (OSError, subprocess.TimeoutExpired):
        pass
    return None


def _ev():
    import torch
    return torch.cuda.Event(enable_timing=True)


def _smi_sample():
    """One amd-smi reading: socket power (W) and the GFX clock of every
    XCD (MHz), or None."""
    import subprocess
    try:
        r = subprocess.run(["amd-smi", "metric", "-p", "-c"], capture_output=True,
                           text=True, timeout=20)
    except (OSError, subprocess.TimeoutExpired):
        return None
    if r.returncode != 0:
        return None
    return parse_smi_metric(r.stdout)


def parse_smi_metric(text):
    """Socket power and per-XCD GFX clocks from the text of `amd-smi metric
    -p -c`: the SOCKET_POWER line, and the CLK line of each section whose
    header (a line like "GFX_3:") names a GFX domain. None without clocks."""
    power, gfx, sec = None, [], None
    for ln in text.splitlines():
        t = ln.strip()
        if t.startswith("SOCKET_POWER:"):
            v = t.split(":", 1)[1].split()[0]
            power = float(v) if v.replace(".", "", 1).isdigit() else None
        elif t.endswith(":") and " " not in t:
            sec = t[:-1]
        elif sec and sec.startswith("GFX") and t.startswith("CLK:"):
            v = t.split(":", 1)[1].split()[0]
            if v.isdigit():
                gfx.append(int(v))
    return {"power_W": power, "gfx_MHz": gfx} if gfx else None


def sustained(fn, seconds, settle=1.0):
    """Run fn (one unit of GPU work, queued) back to back for `seconds`,
    sampling power and clocks from a second thread after `settle` seconds.
    Returns (ms per call over the run, sample summary)."""
    import threading

    import torch
    samples, stop = [], threading.Event()

    def sampler():
        if stop.wait(settle):
            return
        while not stop.is_set():
            s = _smi_sample()
            if s:
                samples.append(s)
            stop.wait(0.2)
    th = threading.Thread(target=sampler)
    n, t_ms = 0, 0.0
    t0 = time.perf_counter()
    th.start()
    while time.perf_counter() - t0 < seconds:
        e0, e1 = _ev(), _ev()
        e0.record()
        for _ in range(20):
            fn()
        e1.record()
        torch.cuda.synchronize()
        n += 20
        t_ms += e0.elapsed_time(e1)
    stop.set()
    th.join()
    clk = sorted(c for s in samples for c in s["gfx_MHz"])
    pw = sorted(s["power_W"] for s in samples if s["power_W"] is not None)
    summ = {"samples": len(samples),
            "gfx_MHz_median": clk[len(clk) // 2] if clk else None,
            "gfx_MHz_min": clk[0] if clk else None, "gfx_MHz_max": clk[-1] if clk else None,
            "socket_power_W_median": pw[len(pw) // 2] if pw else None}
    return t_ms / n, summ


def _operand(rows, cols, half_zero):
    """fp16 N(0, 1) values, with about half of them zero when half_zero (as
    a ReLU output or a ReLU-gated gradient has): on a power-limited GPU the
    MFMA rate depends on how many operand bits toggle."""
    import torch
    a = torch.randn(rows, cols, device="cuda", dtype=torch.float16)
    return a.relu_() if half_zero else a


def _gemm_time(m, n, k, zero_a=False, zero_b=False, reps=20):
    """Median time (s) of a vendor-library fp16 GEMM (torch.matmul, fp32
    accumulation) of [m, k] x [k, n], row-major operands."""
    import torch
    a = _operand(m, k, zero_a)
    b = _operand(k, n, zero_b)
    for _ in range(3):
        torch.matmul(a, b)
    evs = [(_ev(), _ev()) for _ in range(reps)]
    for e0, e1 in evs:
        e0.record()
        torch.matmul(a, b)
        e1.record()
    torch.cuda.synchronize()
    ts = sorted(e0.elapsed_time(e1) for e0, e1 in evs)
    del a, b
    return ts[len(ts) // 2] * 1e-3


SUSTAINED_PASSES = ("E1b.fwd", "E2b.dx", "E1b.dW", "D1T.dW")
STEP_STAT_REPS = 20
NOMINAL_GFX_MHZ = 2400  # the clock the published MFMA peak assumes


MFMA_LOOP_BLOCKS, MFMA_LOOP_ITERS = 512, 60000  # 2 waves per SIMD, ~15 ms a launch


def mfma_loop_bench(seconds=2.0):
    """The library's register-only MFMA loop (fg_mfma_loop, random fp16
    operands about half zero) run back to back: the fp16 MFMA rate this GPU
    sustains with no memory traffic, and its clock and power meanwhile."""
    import torch

    import paper_1909_11150_amd as fg
    out = torch.empty(MFMA_LOOP_BLOCKS * 256, dtype=torch.float32, device="cuda")
    fn = lambda: fg.mfma_loop(out, MFMA_LOOP_BLOCKS, MFMA_LOOP_ITERS)
    for _ in range(3):
        fn()
    torch.cuda.synchronize()
    ms, clk = sustained(fn, seconds)
    work = MFMA_LOOP_BLOCKS * MFMA_LOOP_ITERS * fg.MFMA_LOOP_FLOPS_PER_BLOCK_ITER
    tf = work / ms / 1e9
    return {"tflops": round(tf, 1), "frac_of_peak": round(tf / MFMA_F16_PEAK_TFLOPS, 4),
            "ms_per_launch": round(ms, 3), **clk,
            "measured": f"fg_mfma_loop ({MFMA_LOOP_BLOCKS} workgroups of 4 waves, "
                        f"{MFMA_LOOP_ITERS} iterations of 8 v_mfma_f32_32x32x16_f16 from "
                        f"registers, random fp16 operands about half zero) back to back for "
                        f"{seconds} s"}


def ceiling_bench():
    """The practical MFMA ceiling of this GPU, beside the step:
    - clocks and socket power while the three-stream step runs back to back,
      and while a large vendor-library fp16 GEMM does (dense operands, and
      one operand about half zero as after a ReLU);
    - every convolution pass of the step (alone, one stream, the call's
      whole time) against the vendor GEMM with the pass's output shape and reduction
      length (the GEMM a convolution becomes after an explicit im2col, whose
      own cost is not counted)."""
    import torch

    import synth
    from paper_1909_11150_amd.fcn import Chain
    wl = synth.fcn()
    ch = Chain(wl.layers, wl.weights, wl.x, loss_scale=synth.LOSS_SCALE,
               group_cap_bytes=synth.GROUP_CAP_BYTES)
    target = torch.from_numpy(wl.target).cuda()
    flops_step = sum(3 * L.flops for L in wl.layers)
    prog = ch.program(target, streams=3)
    for _ in range(3):
        prog.run()
    prog.join()

    def step():
        prog.run()
        prog.join()
    ms, clk = sustained(step, 5.0)
    out = {"step": {"ms": round(ms, 4), "tflops": round(flops_step / ms / 1e9, 1),
                    **clk}}
    del prog
    # every pass alone: events around each call (a split pass's reduction
    # included, as the vendor GEMM's own split-K reduction is)
    one = ch.program(target, streams=1)
    conv = [i for i, c in enumerate(one.calls)
            if c.kernel.startswith(("data_conv", "wgrad"))]
    for _ in range(2):
        one.run()
    kev = [{i: (_ev(), _ev()) for i in conv} for _ in range(3)]
    for k in kev:
        one.run(events=k)
    torch.cuda.synchronize()
    ours = {one.calls[i].label: sorted(k[i][0].elapsed_time(k[i][1]) for k in kev)[1] * 1e-3
            for i in conv}
    del one, ch
    torch.cuda.empty_cache()
    ml = mfma_loop_bench(4.0)
    out["mfma_loop"] = {"ms": ml["ms_per_launch"], "tflops": ml["tflops"],
                        **{k: ml[k] for k in ("samples", "gfx_MHz_median", "gfx_MHz_min",
                                              "gfx_MHz_max", "socket_power_W_median")}}
    sq = 8192
    for key, zero_a in (("gemm_8192", False), ("gemm_8192_half_zero_a", True)):
        a = _operand(sq, sq, zero_a)
        b = _operand(sq, sq, False)
        ms_g, clk_g = sustained(lambda: torch.matmul(a, b), 4.0)
        out[key] = {"ms": round(ms_g, 4), "tflops": round(2 * sq ** 3 / ms_g / 1e9, 1),
                    **clk_g}
        del a, b
        torch.cuda.empty_cache()
    rows = []
    for L in wl.layers:
        if L.kind == "conv" and L.w_shape[0] == 1:
            continue  # the K = 1 head runs on vector units
        for pas, shp in (("fwd", L.y_shape), ("dx", L.x_shape), ("dW", None)):
            if shp is None:
                mm, nn = int(np.prod(L.w_shape)) // L.w_shape[0], L.w_shape[0]
            else:
                mm, nn = int(np.prod(shp[:3])), shp[3]
            kk = L.flops // (2 * mm * nn)
            assert 2 * mm * nn * kk == L.flops
            # operands with the pass's zero fractions: the activation (or
            # the gated output gradient) about half zero, the weights dense;
            # the kernel gradient's two operands both about half zero
            t_g = _gemm_time(mm, nn, kk, zero_a=True, zero_b=pas == "dW")
            t_o = ours[f"{L.name}.{pas}"]
            rows.append({"pass": f"{L.name}.{pas}", "gemm_mnk": [mm, nn, kk],
                         "ours_us": round(t_o * 1e6, 1),
                         "ours_tflops": round(L.flops / t_o / 1e12, 1),
                         "gemm_us": round(t_g * 1e6, 1),
                         "gemm_tflops": round(L.flops / t_g / 1e12, 1)})
    out["passes"] = rows
    # four large passes back to back, each alone: the clock each one gets,
    # and its rate against the peak scaled to that clock
    rng = np.random.default_rng(5)
    sus = []
    for label in SUSTAINED_PASSES:
        fn, fl, kern = _op_call(label, rng)
        for _ in range(3):
            fn()
        ms_p, clk_p = sustained(fn, 3.0)
        tf = fl / ms_p / 1e9
        at_clk = (MFMA_F16_PEAK_TFLOPS * clk_p["gfx_MHz_median"] / NOMINAL_GFX_MHZ
                  if clk_p["gfx_MHz_median"] else None)
        sus.append({"pass": label, "kernel": kern, "us": round(ms_p * 1e3, 1),
                    "tflops": round(tf, 1),
                    "frac_of_peak_at_clock": round(tf / at_clk, 3) if at_clk else None,
                    **clk_p})
        del fn
        torch.cuda.empty_cache()
    out["sustained_passes"] = sus
    t_o = sum(r["ours_us"] for r in rows)
    t_g = sum(r["gemm_us"] for r in rows)
    out["passes_total"] = {"ours_us": round(t_o, 1), "gemm_us": round(t_g, 1),
                           "ours_tflops": round(flops_step / t_o / 1e6, 1),
                           "gemm_tflops": round(flops_step / t_g / 1e6, 1)}
    return out


def summarize_ceiling(path):
    with open(path) as f:
        d = json.loads(f.read().strip().splitlines()[-1])
    print("| run | ms per call | TFLOP/s | % of 2.5 PFLOP/s | GFX clock median (min-max), MHz "
          "| socket power median, W | samples |")
    print("|---|---:|---:|---:|---|---:|---:|")
    for k, name in (("step", "encoder-decoder step, 3 streams"),
                    ("mfma_loop", "register-only MFMA loop (fg_mfma_loop), operands about "
                                  "half zero"),
                    ("gemm_8192", "vendor GEMM 8192 x 8192 x 8192, dense N(0,1) operands"),
                    ("gemm_8192_half_zero_a", "the same, A about half zero")):
        if k not in d:
            continue
        v = d[k]
        print(f"| {name} | {v['ms']:.4f} | {v['tflops']:.1f} | "
              f"{100 * v['tflops'] / MFMA_F16_PEAK_TFLOPS:.1f}% | {v['gfx_MHz_median']} "
              f"({v['gfx_MHz_min']}-{v['gfx_MHz_max']}) | {v['socket_power_W_median']} | "
              f"{v['samples']} |")
    if "sustained_passes" in d:
        print()
        print("| pass, back to back | kernel | us per call | TFLOP/s | GFX clock median "
              "(min-max), MHz | socket power median, W | fraction of the peak at that clock |")
        print("|---|---|---:|---:|---|---:|---:|")
        for v in d["sustained_passes"]:
            print(f"| {v['pass']} | `{v['kernel']}` | {v['us']} | {v['tflops']} | "
                  f"{v['gfx_MHz_median']} ({v['gfx_MHz_min']}-{v['gfx_MHz_max']}) | "
                  f"{v['socket_power_W_median']} | {v['frac_of_peak_at_clock']} |")
    print()
    print("| pass | GEMM M x N x K | this library, us | TFLOP/s | vendor GEMM, us | TFLOP/s "
          "| ratio |")
    print("|---|---|---:|---:|---:|---:|---:|")
    for r in d["passes"] + [dict(d["passes_total"], **{"pass": "all 36", "gemm_mnk": None})]:
        mnk = " x ".join(str(v) for v in r["gemm_mnk"]) if r["gemm_mnk"] else ""
        print(f"| {r['pass']} | {mnk} | {r['ours_us']} | {r['ours_tflops']} | "
              f"{r['gemm_us']} | {r['gemm_tflops']} | "
              f"{r['gemm_us'] / r['ours_us']:.2f} |")


def grad_path_bench(reps=20, warmup=3, flush_mib=1024):
    """The gradient path alone on the nine 25 MiB groups of the full
    network's weight gradients (seeded N(0,1) fp16 values): each launch of
    pack, unscale-with-check and unpack is timed with HIP events, after a
    write of flush_mib MiB that evicts the Infinity Cache (256 MB) and the
    L2s, so every byte comes from HBM. Per group and kernel: median and best
    GB/s over `reps`; per kernel: all groups' bytes over the sum of their
    median times. The ceiling is the runtime's own device-to-device copy
    (torch copy_) of each group's fp16 bytes, timed the same way."""
    import torch

    import paper_1909_11150_amd as fg
    import synth
    layers = synth.fcn_layers()
    order = list(reversed(range(len(layers))))
    numels = [layers[i].w_numel for i in order]
    gof, oof, gnum = fg.grad_group_plan(numels, synth.GROUP_CAP_BYTES,
                                        synth.GROUP_ALIGN_BYTES, 2)
    rng = np.random.default_rng(9)
    srcs = [torch.from_numpy(synth.normal(rng, (n,), 1.0)).cuda() for n in numels]
    masters = [torch.empty(n, dtype=torch.float32, device="cuda") for n in numels]
    groups = []
    for g, n in enumerate(gnum):
        mem = [j for j in range(len(numels)) if gof[j] == g]
        groups.append(dict(mem=mem, off=[oof[j] for j in mem], numel=n,
                           g16=torch.empty(n, dtype=torch.float16, device="cuda"),
                           g32=torch.empty(n, dtype=torch.float32, device="cuda"),
                           cpy=torch.empty(n, dtype=torch.float16, device="cuda")))
    flags = torch.zeros(len(groups), dtype=torch.int32, device="cuda")
    flush = torch.empty(flush_mib << 17, dtype=torch.int64, device="cuda")
    kinds = {
        "pack": (4, lambda g, gi: fg.grad_group_pack([srcs[j] for j in g["mem"]],
                                                    g["off"], g["g16"])),
        "unscale": (6, lambda g, gi: fg.grad_unscale_check(
            g["g16"], 1.0 / synth.LOSS_SCALE, g["g32"], flags[gi:gi + 1])),
        "unpack": (8, lambda g, gi: fg.grad_group_unpack(
            g["g32"], [masters[j] for j in g["mem"]], g["off"])),
        "copy_ceiling": (4, lambda g, gi: g["cpy"].copy_(g["g16"])),
    }
    flush.fill_(1)

    def evict():
        # read (not write) the flush buffer: the caches then hold clean
        # lines of it, and the timed launches pay no write-back of them
        flush.max()

    ev = {k: [[] for _ in groups] for k in kinds}
    batch = {k: [] for k in kinds}
    torch.cuda.synchronize()
    for r in range(warmup + reps):
        # all nine groups back to back after one eviction (no byte is read
        # twice within a batch): one event pair per kernel kind
        for k, (_, fn) in kinds.items():
            evict()
            e0, e1 = _ev(), _ev()
            e0.record()
            for gi, g in enumerate(groups):
                fn(g, gi)
            e1.record()
            if r >= warmup:
                batch[k].append((e0, e1))
        # each group alone after its own eviction
        for gi, g in enumerate(groups):
            for k, (_, fn) in kinds.items():
                evict()
                e0, e1 = _ev(), _ev()
                e0.record()
                fn(g, gi)
                e1.record()
                if r >= warmup:
                    ev[k][gi].append((e0, e1))
    torch.cuda.synchronize()
    out = {"method": f"standalone; before each timed batch or launch {flush_mib} MiB "
                     f"are read, evicting the Infinity Cache (256 MB) and the L2s; "
                     f"<kernel>_GBps: the nine groups' launches back to back between "
                     f"one pair of HIP events, median of {reps} reps after {warmup} "
                     f"warm-up; per_group: each launch alone between its own events "
                     f"(event overhead included)",
           "reps": reps, "flush_MiB": flush_mib, "per_group": []}
    for k, (bpe, _) in kinds.items():
        ts = sorted(e0.elapsed_time(e1) * 1e-3 for e0, e1 in batch[k])
        nbytes = bpe * sum(g["numel"] for g in groups)
        out[f"{k}_GBps"] = round(nbytes / ts[len(ts) // 2] / 1e9, 1)
        out[f"{k}_GBps_best"] = round(nbytes / ts[0] / 1e9, 1)
        out[f"{k}_us"] = round(ts[len(ts) // 2] * 1e6, 2)
    for gi, g in enumerate(groups):
        row = {"group": gi, "numel": g["numel"]}
        for k, (bpe, _) in kinds.items():
            ts = sorted(e0.elapsed_time(e1) * 1e-3 for e0, e1 in ev[k][gi])
            med, best = ts[len(ts) // 2], ts[0]
            nbytes = bpe * g["numel"]
            row[k] = {"median_GBps": round(nbytes / med / 1e9, 1),
                      "best_GBps": round(nbytes / best / 1e9, 1),
                      "median_us": round(med * 1e6, 2)}
        out["per_group"].append(row)
    out["size_sweep"] = grad_size_sweep(evict, reps)
    out["pack_frac_hbm"] = round(out["pack_GBps"] / HBM_PEAK_GBPS, 4)
    out["unscale_frac_hbm"] = round(out["unscale_GBps"] / HBM_PEAK_GBPS, 4)
    out["bytes_per_element"] = {"pack": 4, "unscale": 6, "unpack": 8, "copy_ceiling": 4}
    return out


def grad_size_sweep(evict, reps, mib=(4, 8, 16, 32, 64, 128, 256)):
    """Single launches of pack (one member), unscale and the runtime's copy
    on buffers of 4 to 256 MiB of fp16, each after an eviction, HIP events
    around each launch; a least-squares fit of the median times from 16 MiB
    up to t = t0 + bytes / B separates the fixed cost of a launch (t0: the
    launch, the first accesses' latency, the last wave's tail, and the
    events) from the streaming rate B."""
    import torch

    import paper_1909_11150_amd as fg
    n_max = max(mib) << 19
    src = torch.randn(n_max, device="cuda").to(torch.float16)
    dst = torch.empty(n_max, dtype=torch.float16, device="cuda")
    o32 = torch.empty(n_max, dtype=torch.float32, device="cuda")
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    kinds = {
        "pack": (4, lambda n: fg.grad_group_pack([src[:n]], [0], dst[:n])),
        "unscale": (6, lambda n: fg.grad_unscale_check(dst[:n], 2.0 ** -15, o32[:n], flag)),
        "copy_ceiling": (4, lambda n: dst[:n].copy_(src[:n])),
    }
    evs = {(k, m): [] for k in kinds for m in mib}
    for r in range(reps + 2):
        for m in mib:
            for k, (_, fn) in kinds.items():
                evict()
                e0, e1 = _ev(), _ev()
                e0.record()
                fn(m << 19)
                e1.record()
                if r >= 2:
                    evs[(k, m)].append((e0, e1))
    torch.cuda.synchronize()
    out = {"MiB_fp16": list(mib)}
    for k, (bpe, _) in kinds.items():
        med = []
        for m in mib:
            ts = sorted(e0.elapsed_time(e1) * 1e-3 for e0, e1 in evs[(k, m)])
            med.append(ts[len(ts) // 2])
        nbytes = [bpe * (m << 19) for m in mib]
        sel = [i for i, m in enumerate(mib) if m >= 16]
        A = np.array([[1.0, nbytes[i]] for i in sel])
        t0, inv_b = np.linalg.lstsq(A, np.array([med[i] for i in sel]), rcond=None)[0]
        out[k] = {"median_us": [round(t * 1e6, 2) for t in med],
                  "GBps": [round(b / t / 1e9, 1) for b, t in zip(nbytes, med)],
                  "fixed_us": round(t0 * 1e6, 2),
                  "stream_GBps": round(1.0 / inv_b / 1e9, 1),
                  "stream_frac_hbm": round(1.0 / inv_b / 1e9 / HBM_PEAK_GBPS, 4)}
    del src, dst, o32
    return out


def _pass_bytes(L):
    """Minimum HBM bytes of the three passes of a layer (inputs read once,
    output written once, a ReLU-gradient gate read once), fp16."""
    nx, ny, nw = (int(np.prod(L.x_shape)), int(np.prod(L.y_shape)), L.w_numel)
    return [2 * (nx + nw + ny), 2 * (ny + nw + nx), 2 * (nx + ny + nw)]


def _chain_outputs(ch):
    import numpy as np
    return [t.cpu().numpy().view(np.uint16).copy() for t in ch.acts[1:] + ch.g + ch.dw]


def small_configs_bench(steps=50, warmup=5):
    """The single conv, the encoder block and the decoder block (fwd + full
    bwd, one stream), timed with HIP events around each whole pass; each
    against its own roofline: the sum over its ops of max(flops / MFMA
    peak, minimum bytes / HBM peak). These passes are short enough that the
    host's launch calls bound them; the same passes captured once in a HIP
    graph and replayed give the GPU's own time (`graph_*`), after checking
    that every replay reproduces the eager pass bit for bit."""
    import numpy as np
    import torch

    import synth
    from paper_1909_11150_amd.fcn import Chain

    def timed(fn):
        evs = [(_ev(), _ev()) for _ in range(steps)]
        for e0, e1 in evs:
            e0.record()
            fn()
            e1.record()
        torch.cuda.synchronize()
        ts = sorted(e0.elapsed_time(e1) * 1e-3 for e0, e1 in evs)
        return ts[len(ts) // 2], ts[0]

    res = []
    for wl in (synth.single_conv(), synth.encoder_block(), synth.decoder_block()):
        ch = Chain(wl.layers, wl.weights, wl.x)
        ch.set_output_grad(wl.dy)
        flops = sum(3 * L.flops for L in wl.layers)
        roof = 0.0
        for L in wl.layers:
            for b in _pass_bytes(L):
                roof += max(L.flops / (MFMA_F16_PEAK_TFLOPS * 1e12), b / (HBM_PEAK_GBPS * 1e9))

        def step():
            ch.forward()
            ch.backward()
        for _ in range(warmup):
            step()
        med, best = timed(step)
        ref = _chain_outputs(ch)
        # the same pass as a HIP graph, captured on a side stream
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step()
        torch.cuda.current_stream().wait_stream(side)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step()
        same = True
        for _ in range(3):  # replays between eager passes and synchronisations
            for t in ch.acts[1:] + ch.g[:-1] + ch.dw:
                t.zero_()
            g.replay()
            torch.cuda.synchronize()
            same &= all(np.array_equal(a, b) for a, b in zip(ref, _chain_outputs(ch)))
            step()
            torch.cuda.synchronize()
        for _ in range(warmup):
            g.replay()
        gmed, gbest = timed(g.replay)
        res.append({"config": wl.name, "gflop": round(flops / 1e9, 3),
                    "median_us": round(med * 1e6, 2), "best_us": round(best * 1e6, 2),
                    "tflops": round(flops / med / 1e12, 1),
                    "roofline_us": round(roof * 1e6, 2),
                    "frac_of_roofline": round(roof / med, 4),
                    "graph_median_us": round(gmed * 1e6, 2),
                    "graph_tflops": round(flops / gmed / 1e12, 1),
                    "graph_frac_of_roofline": round(roof / gmed, 4),
                    "graph_replays_bit_exact": bool(same)})
        del g, ch
    return res


def main():
    args = parse()
    if args.summarize_stats:
        summarize_stats(args.summarize_stats)
        return
    if args.summarize_pmc:
        summarize_pmc(args.summarize_pmc)
        return
    if args.summarize_mfma:
        summarize_mfma(args.summarize_mfma)
        return
    if args.summarize_ceiling:
        summarize_ceiling(args.summarize_ceiling)
        return
    if args.summarize_trace:
        summarize_trace(args.summarize_trace[0], args.summarize_trace[1],
                        args.launches_per_step, args.steps, args.warmup, args.settle_steps)
        return
    if args.op:
        op_bench(args.op, args.steps, args.warmup)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "the benchmark runs on one GPU only; --gpus must be 1 "
                          "(the library and its step driver implement one GPU's share of "
                          "the data-parallel step; sharding across GPUs is not built)"}))
        sys.exit(2)
    import torch

    import synth
    from paper_1909_11150_amd.fcn import AdamLARS, Chain, LossScaler

    if args.grad_path_only:
        print(json.dumps(grad_path_bench(args.grad_reps)), flush=True)
        return
    if args.ceiling:
        print(json.dumps(ceiling_bench()), flush=True)
        return
    clocks_start = gpu_clocks() if not args.no_clocks else None
    if args.workload == "densenet":
        from paper_1909_11150_amd.densenet import DenseNet
        if args.optimizer or args.zero_copy:
            print(json.dumps({"error": "the dense workload has no zero-copy groups or optimizer"}))
            sys.exit(2)
        # kernel gradients on a second stream (a third stream for the
        # concatenation copies measures slower)
        args.streams = min(args.streams, 2)
        wl = synth.densenet()
        layers = wl.layers
        ch = DenseNet(layers, wl.weights, wl.x, loss_scale=synth.LOSS_SCALE,
                      delta=synth.HUBER_DELTA, group_cap_bytes=synth.GROUP_CAP_BYTES)
    else:
        wl = synth.fcn()
        layers = wl.layers
        opt = dict(optimizer=AdamLARS(), scaler=LossScaler(synth.LOSS_SCALE)) \
            if args.optimizer else {}
        ch = Chain(layers, wl.weights, wl.x, loss_scale=synth.LOSS_SCALE,
                   group_cap_bytes=synth.GROUP_CAP_BYTES, zero_copy=args.zero_copy, **opt)
    target = torch.from_numpy(wl.target).cuda()
    # per-call accounting on one stream, where a call's duration is its own
    prog = ch.program(target, streams=1)
    calls = prog.calls
    torch.cuda.synchronize()
    conv = lambda k: k.startswith(("data_conv", "wgrad", "head_fwd", "head_bwd",
                                   "head_wgrad"))

    for _ in range(args.warmup):
        prog.run()
    torch.cuda.synchronize()

    # detail pass (untimed for `value`): events around every call, and the
    # library's events around every convolution call's main kernel
    det_steps = 2
    det = [{i: (_ev(), _ev()) for i, c in enumerate(calls) if c.fn is not None}
           for _ in range(det_steps)]
    kdet = [{i: (_ev(), _ev()) for i, c in enumerate(calls) if conv(c.kernel)}
            for _ in range(det_steps)]
    for s_ev in det:           # call durations (events around each call)
        prog.run(s_ev)
    for k_ev in kdet:          # main-kernel durations (the library's events)
        prog.run(kernel_events=k_ev)
    torch.cuda.synchronize()
    # per kernel: launches, call ms, work, main-kernel ms (per step)
    per_kernel, per_op = {}, {}
    for s_ev, k_ev in zip(det, kdet):
        for i, (e0, e1) in s_ev.items():
            c = calls[i]
            t = e0.elapsed_time(e1) / det_steps
            tk = k_ev[i][0].elapsed_time(k_ev[i][1]) / det_steps if i in k_ev else t
            k = per_kernel.setdefault(c.kernel, [0, 0.0, 0.0, 0.0])
            k[0] += 1.0 / det_steps
            k[1] += t
            k[2] += c.work / det_steps
            k[3] += tk
            o = per_op.setdefault(c.label, [0.0, c.work, c.kernel, 0.0])
            o[0] += t
            o[3] += tk
    # dominant kernel: the MFMA convolution kernel with the most main-kernel
    # time per step (split variants included: the library's events exclude
    # their reduction launch)
    dom = max((k for k in per_kernel if k.startswith(("data_conv", "wgrad"))),
              key=lambda k: per_kernel[k][3])

    # the timed program: with 3 streams, kernel gradients and the gradient
    # path run beside the input-gradient chain, so a launch of the dominant
    # kernel may share the GPU and its measured duration includes that
    # sharing; `roofline_alone` gives the same kernel's launches in the
    # one-stream detail pass above
    prog = ch.program(target, streams=args.streams)
    calls = prog.calls
    dom_idx = [i for i, c in enumerate(calls) if c.kernel == dom]
    # settle: SETTLE_STEPS steps back to back (about a second) before the
    # warm-up steps; the first steps after the one-stream detail pass run
    # 1-1.4% slower than the steady state a training run is in
    for i in range(args.settle_steps):
        prog.run()
        if i % 10 == 9:
            prog.join()
            torch.cuda.synchronize()
    for _ in range(args.warmup):
        prog.run()
    torch.cuda.synchronize()

    # timed pass: K whole steps; the library's events only around the
    # dominant kernel's launches
    dom_ev = [{i: (_ev(), _ev()) for i in dom_idx} for _ in range(args.steps)]
    for s_ev in dom_ev:          # create the events before the timed region
        for e0, e1 in s_ev.values():
            e0.record()
            e1.record()
    e_start, e_end = _ev(), _ev()
    torch.cuda.synchronize()
    if args.optimizer:
        ch.observe()
        applied0, scale0 = ch.applied, ch.loss_scale
    t0 = time.perf_counter()
    e_start.record()
    for s_ev in dom_ev:
        prog.run(kernel_events=s_ev)
    prog.join()
    e_end.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = e_start.elapsed_time(e_end) / args.steps
    flops_step = sum(3 * L.flops for L in layers)
    value = flops_step / (ms_step * 1e-3) / 1e12

    n_dom = len(dom_idx) * args.steps
    t_dom = sum(e0.elapsed_time(e1) for s_ev in dom_ev for e0, e1 in s_ev.values())
    f_dom = sum(calls[i].work for i in dom_idx) * args.steps
    avg_s = t_dom / n_dom * 1e-3
    achieved = f_dom / n_dom / avg_s / 1e12
    roof = {"bound": "mfma", "kernel": dom, "achieved": round(achieved, 2),
            "peak": MFMA_F16_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": round(achieved / MFMA_F16_PEAK_TFLOPS, 4),
            "avg_launch_us": round(avg_s * 1e6, 2), "launches_per_step": len(dom_idx),
            "flop_per_launch": round(f_dom / n_dom),
            "measured": "HIP events the library records around each launch of the "
                        "kernel (fg_profile_next_launch) inside the timed region, on "
                        "the stream it runs on; a split reduction launched after it "
                        "is not included",
            "traffic": recorded_traffic(dom, args.workload)}
    v = per_kernel[dom]
    alone_s = v[3] / v[0] * 1e-3
    alone = v[2] / v[0] / alone_s / 1e12
    roof_alone = {"kernel": dom, "achieved": round(alone, 2), "unit": "TFLOP/s",
                  "frac": round(alone / MFMA_F16_PEAK_TFLOPS, 4),
                  "avg_launch_us": round(alone_s * 1e6, 2),
                  "measured": "the library's events around each launch in the "
                              "one-stream detail pass of this run (no other kernel "
                              "running)"}
    conv_ms = sum(v[1] for k, v in per_kernel.items() if conv(k))
    conv_main_ms = sum(v[3] for k, v in per_kernel.items() if conv(k))
    _, peak_rate = paper_rates(flops_step / 3, ms_step * 1e-3, conv_ms * 1e-3)

    def bw(name):
        v = per_kernel.get(name)
        return None if not v else round(v[2] / (v[1] * 1e-3) / 1e9, 1)

    out = {
        "metric": "fp16 conv fwd+bwd TFLOP/s per MI355X (% MFMA peak); grad pack GB/s",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic",
        "config": {"workload": WORKLOADS[args.workload],
                   "global_batch": 4, "conv_tflop_per_step": round(flops_step / 1e12, 4),
                   "streams": args.streams, "zero_copy_groups": args.zero_copy,
                   "optimizer": "lars_adam" if args.optimizer else None},
        "mfma_peak_frac": round(value / MFMA_F16_PEAK_TFLOPS, 4),
        "conv_kernels_tflops": round(peak_rate / 1e12, 2),
        "conv_main_kernels_tflops": round(flops_step / (conv_main_ms * 1e-3) / 1e12, 2),
        "conv_rates_measured": "conv_kernels_tflops: step flops over the summed durations "
                               "of the convolution calls (split reductions included) in "
                               "the one-stream detail pass; conv_main_kernels_tflops: over "
                               "the summed main-kernel durations (no split reductions)",
        "grad_pack_GBps_in_step": bw("copy_pieces_kernel<2>"),
        "grad_unscale_GBps_in_step": bw("unscale_vec_kernel"),
        "grad_unpack_GBps_in_step": bw("copy_pieces_kernel<4>"),
        "wall_s_timed": round(wall, 3),
        "settle_steps_before_warmup": args.settle_steps,
        "roofline": roof,
        "roofline_alone": roof_alone,
    }
    if args.optimizer:
        ch.observe()
        nrm = [v for k, v in per_op.items() if k.endswith(".norms")]
        aps = [v for k, v in per_op.items() if k.endswith(".apply")]
        ap = (sum(v[0] for v in aps), sum(v[1] for v in aps))
        n_ms, n_b = sum(v[0] for v in nrm), sum(v[1] for v in nrm)
        out["optimizer"] = {
            "norms_ms": round(n_ms, 4), "norms_GBps": round(n_b / (n_ms * 1e-3) / 1e9, 1),
            "apply_ms": round(ap[0], 4), "apply_GBps": round(ap[1] / (ap[0] * 1e-3) / 1e9, 1),
            "gradients": "fp16 group slots" if args.zero_copy else "fp32 unpacked",
            "bytes_per_param": "norms: w, m, v, gradient read; apply: the same read, "
                               "w, m, v, fp16 copy written",
            "apply_overlap": "per layer, beside the next step's forward pass",
            "timed_updates_applied": ch.applied - applied0,
            "loss_scale_start": scale0, "loss_scale_end": ch.loss_scale}
    # spread of single steps, after the timed region: each step between its
    # own events on the main stream, its side streams joined before the end
    # event (so no step overlaps the next, unlike the timed region's)
    per_step = []
    for _ in range(STEP_STAT_REPS):
        e0, e1 = _ev(), _ev()
        e0.record()
        prog.run()
        prog.join()
        e1.record()
        per_step.append((e0, e1))
    torch.cuda.synchronize()
    st = sorted(e0.elapsed_time(e1) for e0, e1 in per_step)
    out["step_ms_stats"] = {
        "reps": STEP_STAT_REPS, "median": round(st[len(st) // 2], 4),
        "min": round(st[0], 4), "max": round(st[-1], 4),
        "measured": "after the timed region: single steps, each between its own HIP "
                    "events with its side streams joined, so no step overlaps the next"}
    under_load = None
    if not args.no_clocks:
        # clocks and power while the timed program runs back to back (after
        # the timed region, which is too short to sample)
        def one_step():
            prog.run()
            prog.join()
        ms_sus, under_load = sustained(one_step, 2.5, settle=0.5)
        under_load = {"ms_per_step": round(ms_sus, 4), **under_load}
    if args.detail:
        det = {"per_kernel": {k: {"launches_per_step": v[0], "ms_per_step": v[1],
                                  "work_per_step": v[2], "main_kernel_ms_per_step": v[3]}
                              for k, v in per_kernel.items()},
               "per_op": {k: {"ms": v[0], "main_kernel_ms": v[3],
                              "rate": v[1] / (v[3] * 1e-3) / 1e12,
                              "kernel": v[2]} for k, v in per_op.items()}}
        with open(args.detail, "w") as f:
            json.dump(det, f, indent=1)
    del prog, ch
    torch.cuda.empty_cache()
    if args.workload == "fcn" and not args.no_extras:
        # the gradient path alone, caches flushed (the grad-pack GB/s of the
        # metric), and the three small configurations against their rooflines
        gp = grad_path_bench(args.grad_reps)
        out["grad_pack_GBps"] = gp["pack_GBps"]
        out["grad_unscale_GBps"] = gp["unscale_GBps"]
        out["grad_unpack_GBps"] = gp["unpack_GBps"]
        out["grad_path"] = gp
        out["small_configs"] = small_configs_bench()
        ml = mfma_loop_bench()
        out["mfma_loop"] = ml
        out["value_frac_of_mfma_loop"] = round(out["value"] / ml["tflops"], 4)
    if not args.no_clocks:
        out["clocks"] = {"start": clocks_start, "end": gpu_clocks(),
                         "under_load": under_load,
                         "note": "start and end are idle readings; under_load samples "
                                 "amd-smi while the timed step runs back to back for "
                                 "2.5 s (the chip is power-limited: its GFX clock sits "
                                 "below the 2.4 GHz the MFMA peak assumes)"}
    if not args.no_cpu:
        cb = cpu_baseline(layers, args.cpu_seconds)
        cb["cpu_model"] = cpu_model()
        if args.workload == "fcn":
            cb["grad_path"] = cpu_grad_baseline(args.cpu_seconds / 4)
        out["cpu_baseline"] = cb
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

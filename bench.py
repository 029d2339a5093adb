"""Benchmark of the fused Winograd 3x3 convolution on one MI355X.

A step is one wino_conv_run of the VGG-style layer N=32, C=K=64, 224x224,
F(4x4,3x3): the kernel transform followed by the fused kernel (input transform,
per-frequency products on the matrix cores, output transform).  Inputs are
seeded synthetic tensors already resident in device memory.

The metric is the effective rate, direct-convolution flops (2*N*C*K*H*W*9) per
second.  The JSON line also carries the fused kernel's own rate against the
fp32 matrix-core roofline (transform-domain flops 2*T^2*tiles*C*K over the
kernel's mean duration: K back-to-back calls of it alone between two HIP events
on the stream it runs on, queued right behind the timed steps), the
three-stage variant's step time on the same layer, a per-layer table of every
configured (layer, m) pair ("layers": fused and three-stage call and kernel
times, matrix-core and HBM fractions of the kernels), per layer the tile size,
algorithm and blocking a per-layer tuning picks, timed the same way
("tuned_layers"), and the CPU oracle timed on the host cores.  Before the W
warm-up steps of every measurement, the step runs untimed for about 150 ms
("settle_ms") so that the shader clock has reached its steady level (it ramps up
over the first tens of milliseconds of load).

    python bench.py [--steps K] [--warmup W] [--layer ID --m M] [--all] [--no-cpu] [--no-layers]

--all adds a per-(layer, m, algorithm) table (stderr, and --out): back-to-back step
time, the median of single calls warm and cold (a 512 MB scratch write before each
cold call evicts L2 and the Infinity Cache), and the transform-domain kernel time;
plus, per layer, the m, blocking and algorithm a tuned plan picks (algo "tuned"),
each fused blocking the library is built for at the layer's tile sizes (algo
"fused_R<r>_K<k>"), and on layers with C >= 128 the fused kernel with every work
item split into 2 and 4 channel pieces (algo "fused_csplitP"); and per layer the
FFT-tile algorithm (algo "fft", 16 x 16 tiles; its "transform-domain" rate counts
the real flops of its complex products) and the three-stage F(7x7,3x3); and for the
launch-bound 56x56 layer at F(2) one call captured in a HIP graph and replayed
(algo "fused_graph").
"""

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

P_MFMA_F32 = 157.3e12   # MI355X dense fp32 matrix peak, FLOP/s
B_HBM = 8.0e12          # MI355X HBM3E peak, B/s
# the sources the fused kernel is built from (its counters, taken on another
# version of them, no longer describe it)
KERNEL_SRCS = [os.path.join(ROOT, "paper_1912_02165_amd", "csrc", f) for f in
               ("wino_ws.h", "wino_device.h", "wino_transforms.h", "wino_fused_inst.hip")]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--layer", type=int, default=2)
    ap.add_argument("--m", type=int, default=4)
    ap.add_argument("--all", action="store_true", help="also time every (layer, m, algorithm)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-layers", action="store_true", help="skip the per-layer table")
    ap.add_argument("--out", default=None, help="append the per-pair table (JSON lines) here")
    return ap.parse_args()


def kernel_source_hash():
    h = hashlib.sha256()
    for path in KERNEL_SRCS:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel, workload):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they were taken
    on the current kernel source; else None."""
    try:
        with open(TRAFFIC_FILE) as f:
            entries = json.load(f)
    except (OSError, ValueError):
        return None
    for e in entries:
        if (e.get("kernel") == kernel and e.get("workload") == workload
                and e.get("source_hash") == kernel_source_hash()):
            return e.get("bytes_per_launch")
    return None


SETTLE_MS = 150.0
# Back-to-back timings cover at least this much GPU time (at most MAX_TIMED_CALLS calls).
MIN_TIMED_MS = 3.0
MAX_TIMED_CALLS = 4096


def settle(call, ms=SETTLE_MS):
    """Runs `call` back to back until about `ms` of GPU time has passed (untimed).
    The shader clock ramps up over the first tens of milliseconds of load (a 224x224
    layer's kernel measures 5-10 % slower in its first 20 ms); this keeps every
    measurement at the steady clock a serving loop runs at."""
    import torch
    t0 = time.perf_counter()
    n = 0
    while True:
        for _ in range(4):
            call()
        n += 4
        torch.cuda.synchronize()
        if (time.perf_counter() - t0) * 1e3 >= ms or n >= 4096:
            return n


def rep_times(p, x, w, y, steps, stream, scratch=None):
    """Per-call times (ms) of `steps` separate run() calls, each bracketed by its own
    events; with `scratch`, the buffer is overwritten before every call (outside the
    events) so that the call finds neither L2 nor the Infinity Cache warm."""
    import torch
    times = []
    for _ in range(steps):
        if scratch is not None:
            scratch.fill_(1.0)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        p.run(x, w, y)
        b.record(stream)
        b.synchronize()
        times.append(a.elapsed_time(b))
    return sorted(times)[len(times) // 2]


def per_call_ms(timed, steps, exact=False):
    """Mean ms per call of back-to-back calls between two events (per-call events
    would add a dispatch gap to every call, several microseconds against the
    smallest layers' kernels).  `timed(n)` queues n calls between two events and
    returns the elapsed ms; it is called for `steps` calls and, unless `exact`,
    once more with enough calls to cover MIN_TIMED_MS (at most MAX_TIMED_CALLS)
    when those took less.  Each window is queued behind untimed calls of the same
    kind with no host synchronisation between, so that the shader clock, which
    falls within a millisecond or so of idling and takes tens of milliseconds to
    rise again, is where the previous phase left it."""
    ms = timed(steps)
    if exact or ms >= MIN_TIMED_MS:
        return ms / steps
    n = min(MAX_TIMED_CALLS, max(steps, int(MIN_TIMED_MS / max(ms / steps, 1e-4)) + 1))
    return timed(n) / n


def time_pair(layer, m, algo, steps, warmup, x, w, per_call=False, tuning=None, exact=False):
    """Time `steps` steps; returns dict with ms_per_step and the transform-domain
    kernel's average duration (ms) measured between events on the same stream.
    Every back-to-back timing covers at least MIN_TIMED_MS of GPU time (more calls
    than `steps` for small layers, so that the first dispatch's latency does not
    weigh on the mean), except the whole steps when `exact` is set: those are then
    exactly `steps` calls.
    per_call: also the median time of single calls, warm and cold (after a 512 MB
    scratch write that evicts L2 and the 256 MB Infinity Cache)."""
    import torch
    import paper_1912_02165_amd as wc
    N, C, K, H, W = layer.N, layer.C, layer.K, layer.H, layer.W
    y = torch.empty((N, K, H, W), dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    with wc.Plan(N, C, K, H, W, m, algo, tuning) as p:
        settle(lambda: p.run(x, w, y))
        for _ in range(warmup):
            p.run(x, w, y)
        torch.cuda.synchronize()

        # n back-to-back calls between two events, behind `pre` untimed ones
        def window(call, n, pre):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            for _ in range(pre):
                call()
            a.record(stream)
            for _ in range(n):
                call()
            b.record(stream)
            torch.cuda.synchronize()
            return a.elapsed_time(b)

        def back_to_back(call, exact_count=False, pre=0):
            return per_call_ms(lambda n: window(call, n, pre), steps, exact_count)

        # whole steps, then the two phases of a step timed apart: the
        # transform-domain kernels on the pretransformed kernels (right after the
        # steps, behind a few of their calls), then the kernel transform
        torch.cuda.synchronize()
        ms_step = back_to_back(lambda: p.run(x, w, y), exact)
        body_ms = back_to_back(lambda: p.run_pretransformed(x, y), pre=max(4, warmup))
        wt_ms = back_to_back(lambda: p.set_weights(w))
        nt, dflops, tflops = p.info()
        p.status()
        res = {"ms_per_step": ms_step, "weight_transform_ms": wt_ms, "body_ms": body_ms,
               "direct_flops": dflops, "tdomain_flops": tflops, "tiles": nt,
               "kernel": p.describe(), "params": p.params()}
        if per_call:
            res["warm_call_ms_median"] = rep_times(p, x, w, y, steps, stream)
            scratch = torch.empty(128 << 20, dtype=torch.float32, device="cuda")
            res["cold_call_ms_median"] = rep_times(p, x, w, y, steps, stream, scratch)
            del scratch
    return res


def time_graph(layer, m, steps, warmup, x, w):
    """One wino_conv_run captured in a HIP graph (torch.cuda.CUDAGraph), replayed:
    back-to-back ms per replay and the median of separately timed replays."""
    import torch
    import paper_1912_02165_amd as wc
    N, C, K, H, W = layer.N, layer.C, layer.K, layer.H, layer.W
    y = torch.empty((N, K, H, W), dtype=torch.float32, device="cuda")
    with wc.Plan(N, C, K, H, W, m, "fused") as p:
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            for _ in range(warmup):
                p.run(x, w, y)
        torch.cuda.current_stream().wait_stream(s)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            p.run(x, w, y)
        for _ in range(warmup):
            g.replay()
        torch.cuda.synchronize()
        stream = torch.cuda.current_stream()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(steps):
            g.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        ms_step = e0.elapsed_time(e1) / steps
        single = []
        for _ in range(steps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            g.replay()
            b.record(stream)
            torch.cuda.synchronize()
            single.append(a.elapsed_time(b))
        del g
    return ms_step, sorted(single)[len(single) // 2]


def algorithmic_bytes(layer, m, algo, kit=64):
    """Minimal HBM bytes of the transform-domain part of one call: the fused kernel
    reads x and the transformed kernels W' and writes y; the three-stage pipeline
    also writes and reads U (T^2 x tiles x C) and M (T^2 x tiles x K)."""
    T2 = (m + 2) ** 2
    tiles = layer.N * -(-layer.H // m) * -(-layer.W // m)
    x = 4 * layer.N * layer.C * layer.H * layer.W
    y = 4 * layer.N * layer.K * layer.H * layer.W
    wt = 4 * T2 * layer.C * layer.K
    if algo == "fused":
        return x + y + wt
    return x + 2 * 4 * T2 * tiles * layer.C + wt + 2 * 4 * T2 * tiles * layer.K + y


def layer_table(steps=20, warmup=10):
    """Every configured (layer, m) pair, fused and three-stage: call time, kernel
    (transform-domain) time, and the kernels' fractions of the fp32 matrix peak
    and of the HBM peak (algorithmic bytes over kernel time)."""
    import torch
    from paper_1912_02165_amd import workloads
    rows = []
    for lay in workloads.LAYERS:
        xn, wn = workloads.layer_inputs(lay)
        xa, wa = torch.from_numpy(xn).cuda(), torch.from_numpy(wn).cuda()
        del xn, wn
        for m in lay.ms:
            row = {"workload": lay.tag(m)}
            for algo in ("fused", "three_stage"):
                r = time_pair(lay, m, algo, steps, warmup, xa, wa)
                ms = r["body_ms"] * 1e-3
                row[algo] = {
                    "ms_per_call": r["ms_per_step"],
                    "kernel_ms": r["body_ms"],
                    "eff_tflops": r["direct_flops"] / (r["ms_per_step"] * 1e-3) / 1e12,
                    "mfma_frac": r["tdomain_flops"] / ms / P_MFMA_F32,
                    "hbm_frac": algorithmic_bytes(lay, m, algo) / ms / B_HBM,
                    "kernel": r["kernel"],
                }
            row["fused_speedup_over_three_stage"] = (row["three_stage"]["kernel_ms"]
                                                     / row["fused"]["kernel_ms"])
            rows.append(row)
            print(json.dumps(row), file=sys.stderr, flush=True)
        del xa, wa
    return rows


def tuned_table(steps=20, warmup=10):
    """Per configured layer, the tile size, algorithm and blocking the per-layer
    tuning picks (`wino_conv_plan_tuned` over every built fused blocking at F(2),
    F(4), F(5), F(6) and the three-stage pipeline at those and F(7)), timed like
    the pairs of `layer_table`."""
    import torch
    import paper_1912_02165_amd as wc
    from paper_1912_02165_amd import workloads
    rows = []
    for lay in workloads.LAYERS:
        xn, wn = workloads.layer_inputs(lay)
        xa, wa = torch.from_numpy(xn).cuda(), torch.from_numpy(wn).cuda()
        del xn, wn
        tp = wc.Plan.tuned(lay.N, lay.C, lay.K, lay.H, lay.W, wc.WINO_TUNE_ALL_M | wc.WINO_TUNE_THREE_STAGE)
        m, algo = tp.m, tp.algo
        _, _, R, kit = tp.params()
        tp.close()
        tuning = {"tiles_per_wg": R, "k_per_wg": kit} if algo == "fused" else None
        r = time_pair(lay, m, algo, steps, warmup, xa, wa, tuning=tuning)
        ms = r["body_ms"] * 1e-3
        row = {"workload": lay.tag(m), "m": m, "algo": algo, "tiles_per_wg": R, "k_per_wg": kit,
               "ms_per_call": r["ms_per_step"], "kernel_ms": r["body_ms"],
               "eff_tflops": r["direct_flops"] / (r["ms_per_step"] * 1e-3) / 1e12,
               "eff_tflops_kernel": r["direct_flops"] / ms / 1e12,
               "mfma_frac": r["tdomain_flops"] / ms / P_MFMA_F32, "kernel": r["kernel"]}
        rows.append(row)
        print(json.dumps(row), file=sys.stderr, flush=True)
        del xa, wa
    return rows


def host_cpu():
    """(nproc, CPU model name) of the host."""
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return os.cpu_count(), model


def cpu_baseline(layer, budget_s=20.0):
    """The oracle (plain C direct convolution, fp64 accumulation, OpenMP) on the first
    images of the layer: one image to size the sample, then as many images as fit in
    about budget_s seconds (at most the whole layer)."""
    from paper_1912_02165_amd import workloads
    from oracle import direct
    x1, w = workloads.layer_inputs(layer, n_images=1)
    t = time.perf_counter()
    direct.direct_conv(x1, w)
    t1 = time.perf_counter() - t
    n = max(1, min(layer.N, int(budget_s / max(t1, 1e-3))))
    if n > 1:
        xs, w = workloads.layer_inputs(layer, n_images=n)
        t = time.perf_counter()
        direct.direct_conv(xs, w)
        dt = time.perf_counter() - t
    else:
        dt = t1
    flops = layer.direct_flops / layer.N * n
    nproc, model = host_cpu()
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": direct.num_threads(),
            "nproc": nproc, "cpu_model": model, "kind": "oracle",
            "sample": f"{n} of {layer.N} images of {layer.name} (direct conv, fp64 accumulation), "
                      f"{dt:.2f} s"}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              "(the convolution shards over images with no exchange; see the design notes)",
              file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_1912_02165_amd import workloads

    layers = None if args.no_layers else layer_table()
    tuned = None if args.no_layers else tuned_table()
    layer = workloads.LAYER_BY_ID[args.layer]
    m = args.m
    x_np, w_np = workloads.layer_inputs(layer)
    x = torch.from_numpy(x_np).cuda()
    w = torch.from_numpy(w_np).cuda()

    fused = time_pair(layer, m, "fused", args.steps, args.warmup, x, w, exact=True)
    three = time_pair(layer, m, "three_stage", args.steps, args.warmup, x, w, exact=True)

    kernel_ms = fused["body_ms"]
    achieved = fused["tdomain_flops"] / (kernel_ms * 1e-3)
    workload = layer.tag(m)
    traffic = measured_traffic("fused", workload)
    rec = {
        "metric": "effective TFLOP/s per conv layer (direct-conv FLOPs) + % of MFMA/HBM roofline",
        "value": fused["direct_flops"] / (fused["ms_per_step"] * 1e-3) / 1e12,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": fused["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": workload, "N": layer.N, "C": layer.C, "K": layer.K, "H": layer.H,
                   "W": layer.W, "m": m, "algo": "fused", "stride": 1, "pad": 1},
        "roofline": {"bound": "mfma", "achieved": achieved / 1e12, "peak": P_MFMA_F32 / 1e12,
                     "unit": "TFLOP/s", "frac": achieved / P_MFMA_F32, "traffic": traffic,
                     "kernel": fused["kernel"], "kernel_ms": kernel_ms,
                     "kernel_ms_timing": "HIP events around `steps` back-to-back run_pretransformed "
                                         "calls on its stream, mean per call"},
        "tdomain_tflops_per_step": fused["tdomain_flops"] / (fused["ms_per_step"] * 1e-3) / 1e12,
        "weight_transform_ms": fused["weight_transform_ms"],
        "three_stage": {"ms_per_step": three["ms_per_step"],
                        "value": three["direct_flops"] / (three["ms_per_step"] * 1e-3) / 1e12,
                        "body_ms": three["body_ms"]},
        "cpu_baseline": None,
        "settle_ms": SETTLE_MS,
        "layers": layers,
        "tuned_layers": tuned,
    }
    if not args.no_cpu:
        rec["cpu_baseline"] = cpu_baseline(layer)

    if args.all:
        import paper_1912_02165_amd as wc
        rows = []
        tuned_done = set()
        fft_done = set()
        for lay, mm in workloads.PAIRS:
            xn, wn = workloads.layer_inputs(lay)
            xa, wa = torch.from_numpy(xn).cuda(), torch.from_numpy(wn).cuda()
            cases = [(mm, "fused", "fused"), (mm, "three_stage", "three_stage")]
            # every built fused blocking at this tile size
            cases += [(mm, "fused", "fused_R%d_K%d" % (R, kit))
                      for (bm, R, kit) in wc.wino_fused_blockings() if bm == mm]
            tuned_blocking = None
            if lay.id not in tuned_done:
                # the tile size, blocking and algorithm a per-layer tuning picks (timed now)
                tuned_done.add(lay.id)
                tp = wc.Plan.tuned(lay.N, lay.C, lay.K, lay.H, lay.W,
                                   wc.WINO_TUNE_ALL_M | wc.WINO_TUNE_THREE_STAGE)
                _, _, tR, tkit = tp.params()
                tuned_blocking = (tR, tkit)
                cases.append((tp.m, tp.algo, "tuned"))
                tp.close()
            if lay.C >= 128:
                # every work item split into channel pieces (partial outputs added)
                cases += [(mm, "fused", "fused_csplit%d" % P) for P in (2, 4)]
            if lay.id not in fft_done:
                # the FFT-tile algorithm (16 x 16 tiles, m = 14) and the three-stage
                # F(7x7,3x3), once per layer
                fft_done.add(lay.id)
                cases.append((14, "fft", "fft"))
                cases.append((7, "three_stage", "three_stage"))
            for m_c, algo, label in cases:
                tuning = None
                if label.startswith("fused_csplit"):
                    tuning = {"channel_splits": int(label[len("fused_csplit"):])}
                elif label.startswith("fused_R"):
                    R, kit = (int(v) for v in label[len("fused_R"):].split("_K"))
                    tuning = {"tiles_per_wg": R, "k_per_wg": kit}
                elif label == "tuned" and algo == "fused":
                    tuning = {"tiles_per_wg": tuned_blocking[0], "k_per_wg": tuned_blocking[1]}
                r = time_pair(lay, m_c, algo, args.steps, args.warmup, xa, wa, per_call=True,
                              tuning=tuning)
                wl = lay.name + "/FFT(16x16 tiles)" if algo == "fft" else lay.tag(m_c)
                row = {"workload": wl, "algo": label, "ms_per_step": r["ms_per_step"],
                       "eff_tflops": r["direct_flops"] / (r["ms_per_step"] * 1e-3) / 1e12,
                       "warm_call_ms_median": r["warm_call_ms_median"],
                       "cold_call_ms_median": r["cold_call_ms_median"],
                       "eff_tflops_cold": r["direct_flops"] / (r["cold_call_ms_median"] * 1e-3) / 1e12,
                       "body_ms": r["body_ms"],
                       "tdomain_tflops_body": r["tdomain_flops"] / (r["body_ms"] * 1e-3) / 1e12,
                       "mfma_frac_body": r["tdomain_flops"] / (r["body_ms"] * 1e-3) / P_MFMA_F32,
                       "weight_transform_ms": r["weight_transform_ms"]}
                row["kernel"] = r["kernel"]
                if label == "tuned":
                    row["tuned_choice"] = {"m": m_c, "algo": algo,
                                           "tiles_per_wg": tuned_blocking[0] if algo == "fused" else 0,
                                           "k_per_wg": tuned_blocking[1] if algo == "fused" else 0}
                rows.append(row)
                print(json.dumps(row), file=sys.stderr, flush=True)
            if lay.id == 1 and mm == 2:
                # the launch-bound layer as a replayed HIP graph of one call
                g_step, g_single = time_graph(lay, mm, args.steps, args.warmup, xa, wa)
                row = {"workload": lay.tag(mm), "algo": "fused_graph", "ms_per_step": g_step,
                       "eff_tflops": lay.direct_flops / (g_step * 1e-3) / 1e12,
                       "warm_call_ms_median": g_single}
                rows.append(row)
                print(json.dumps(row), file=sys.stderr, flush=True)
            del xa, wa
        if args.out:
            with open(args.out, "a") as f:
                for row in rows:
                    f.write(json.dumps(row) + "\n")
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()

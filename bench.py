"""Benchmark: PointNet++ SSG classifier forward, batch 32 x 1024 points,
delayed aggregation, on one MI355X (--workload picks any of the five
synthetic workloads instead).

One step = one full forward of the batch (FPS, ball query, per-point MLP,
aggregation for both set-abstraction levels, group-all MLP, FC head).
Inputs and weights are resident in HBM before timing; the timed steps
replay HIP graphs of the two-stream forward; independent batches may be
kept in flight on separate streams (the count that gives the highest
throughput among 1-4 is used and reported, with the single-batch latency
and its per-step distribution).
The JSON line also carries:
  - conventional: the same network in the original order (Eq. (1)) on the
    GPU and the delayed/conventional speedup;
  - limited_order: the limited delayed aggregation of Sec. 7.3 (only the
    first layer's product hoisted; exact) and its speedup over the
    conventional order;
  - stages: per-kernel-call durations from HIP events on the stream each
    kernel runs on (an eager pass over the same steps), with each call's
    algorithmic work derived from its arguments;
  - roofline: the dominant kernel's achieved rate against MI355X peak;
  - cpu_baseline: the CPU oracle timed on this host (single thread, all
    cores, and the conventional forward).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "clouds/sec end-to-end + centroids/sec per module; % HBM and MFMA peak"
WORKLOAD = "pointnet2_cls"
DESCRIBE = {
    "sa_module": "one set-abstraction module, 1024 -> 512 centroids, K 32, 3 -> 64 -> 64 -> 128",
    "pointnet2_cls": "PointNet++ SSG classifier",
    "dgcnn": "DGCNN, 4 EdgeConv layers with k = 20 in feature space, 1x1 conv to 1024, global max",
    "pointnet2_seg": "PointNet++ SSG segmentation of indoor rooms, 4 SA levels, 4 FP levels",
    "lidar": "3-level PointNet++ backbone on 16384-point LiDAR sweeps, bf16 MLPs",
}
HBM_PEAK_GBS = 8000.0
MFMA_F32_PEAK_TFLOPS = 157.3
MFMA_BF16_PEAK_TFLOPS = 2516.6
N_CUS = 256   # MI355X compute units (the ALU peak is spread evenly over them)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=500)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default=WORKLOAD)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--eager", action="store_true", help="time eager launches instead of graph replay")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a plain 256 MiB device copy (reference for HBM counters)")
    return ap.parse_args()


# ----------------------------------------------------------------------------
# per-call event timing (eager pass)
# ----------------------------------------------------------------------------

class StageTimer:
    """Wraps the ops entry points so every call records a start/end event on
    the stream it is launched on."""

    NAMES = ("fps", "ball_query", "knn", "pointwise_mlp", "aggregate_max", "conventional_module", "interpolate3")

    def __init__(self, ops):
        import torch
        self.torch = torch
        self.ops = ops
        self.orig = {n: getattr(ops, n) for n in self.NAMES}
        self.records = []     # (name#k, start, end)
        self.work = {}        # name#k -> (bound, amount, extra)
        self.counts = {}
        self.active = False

    def install(self):
        torch = self.torch
        for n, fn in self.orig.items():
            def wrap(*a, __n=n, __fn=fn, **kw):
                if not self.active:
                    return __fn(*a, **kw)
                k = self.counts.get(__n, 0)
                self.counts[__n] = k + 1
                s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                s.record()
                r = __fn(*a, **kw)
                e.record()
                self.records.append((f"{__n}#{k}", s, e))
                self.work[f"{__n}#{k}"] = call_work(__n, a, kw)
                return r
            setattr(self.ops, n, wrap)

    def uninstall(self):
        for n, fn in self.orig.items():
            setattr(self.ops, n, fn)

    def begin_step(self):
        self.counts = {}

    def summary(self):
        self.torch.cuda.synchronize()
        acc = {}
        for name, s, e in self.records:
            acc.setdefault(name, []).append(s.elapsed_time(e))
        return {k: float(np.mean(v)) for k, v in acc.items()}


# ----------------------------------------------------------------------------
# algorithmic work of one call, from its arguments (documented in the design doc)
# ----------------------------------------------------------------------------

def call_work(name, a, kw):
    """(bound, amount, extra) for one entry-point call; amount in TFLOP
    (alu / mfma) or GB (hbm).

    fps:            (M-1) * N point updates per cloud, 8 flops each (3 sub,
                    1 mul, 2 fma) -> alu
    ball_query:     B * M * N candidate tests (upper bound; early exit scans
                    fewer), 8 flops each -> alu; its compulsory HBM bytes
                    (points, centroids, NIT and counts) reported beside it
    knn:            B * M * N pairs, 3 * C flops each (sub, mul, add) -> alu;
                    compulsory bytes (reference and query rows, NIT) beside it
    pointwise_mlp:  2 * rows * sum(C_l * C_l+1) -> mfma
    aggregate_max:  compulsory HBM bytes -- every PFT row read once, the NIT,
                    the centroid indices or rows, the output -> hbm (the
                    bytes of the gathered rows are reported beside it)
    conventional:   2 * B*M*K * sum(C_l * C_l+1) -> mfma
    interpolate3:   B * Nd * Ns pairs, 8 flops each -> alu
    """
    def arg(i, key, default=None):
        return a[i] if len(a) > i else kw.get(key, default)

    if name == "fps":
        xyz, M = arg(0, "xyz"), arg(1, "M")
        B, N = xyz.shape[0], xyz.shape[1]
        # one workgroup per cloud walks M - 1 dependent iterations
        return ("alu", 8.0 * B * (M - 1) * N / 1e12, {"serial_iterations": M - 1, "workgroups": B})
    if name == "ball_query":
        xyz, q, K = arg(0, "xyz"), arg(1, "qxyz"), arg(3, "K")
        B, N, M = xyz.shape[0], xyz.shape[1], q.shape[1]
        comp = 12 * B * N + 12 * B * M + 4 * B * M * K + 4 * B * M
        return ("alu", 8.0 * B * M * N / 1e12, {"compulsory_bytes": comp})
    if name == "knn":
        ref, q, K = arg(0, "ref"), arg(1, "query"), arg(2, "K")
        B, N, C = ref.shape
        M = q.shape[1]
        comp = 4 * B * N * C + (0 if q.data_ptr() == ref.data_ptr() else 4 * B * M * C) + 4 * B * M * K
        return ("alu", 3.0 * C * B * M * N / 1e12, {"compulsory_bytes": comp})
    if name == "pointwise_mlp":
        x0, prm = arg(0, "x0"), arg(1, "p")
        rows = int(np.prod(x0.shape[:-1]))
        d = prm.dims
        return ("mfma", 2.0 * rows * sum(x * y for x, y in zip(d[:-1], d[1:])) / 1e12, None)
    if name == "aggregate_max":
        pft, nit = arg(0, "pft"), arg(1, "nit")
        cidx, cfeat, out = arg(2, "cidx"), arg(3, "cfeat"), kw.get("out")
        B, N = pft.shape[0], pft.shape[1]
        M, K = nit.shape[1], nit.shape[2]
        C = out.shape[-1] if out is not None else pft.shape[-1]
        s = pft.element_size()
        comp = B * N * C * s + 4 * B * M * K + 4 * B * M * C
        if cidx is not None:
            comp += 4 * B * M
        if cfeat is not None:
            comp += B * M * C * s
        return ("hbm", comp / 1e9, {"logical_gather_bytes": B * M * K * C * s})
    if name == "conventional_module":
        nit, prm = arg(0, "nit"), arg(1, "p")
        rows = int(np.prod(nit.shape))
        d = prm.dims
        return ("mfma", 2.0 * rows * sum(x * y for x, y in zip(d[:-1], d[1:])) / 1e12, None)
    if name == "interpolate3":
        dst, src = arg(0, "xyz_dst"), arg(1, "xyz_src")
        return ("alu", 8.0 * dst.shape[0] * dst.shape[1] * src.shape[1] / 1e12, None)
    return None


PEAKS = {"alu": (157.3, "TFLOP/s"), "mfma": (MFMA_F32_PEAK_TFLOPS, "TFLOP/s"), "hbm": (HBM_PEAK_GBS, "GB/s")}


def load_traffic(kernel_key):
    """HBM bytes per launch measured with rocprofv3 FETCH_SIZE / WRITE_SIZE,
    recorded in profiles/pmc_traffic.txt together with a hash of the kernel's
    source file; None if absent or if the source has changed since."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "pmc_traffic.txt")
    if not os.path.exists(path):
        return None
    for line in open(path):
        f = line.split()
        if len(f) >= 5 and not line.startswith("#") and f[0] == kernel_key:
            src = os.path.join(ROOT, "paper_2008_06967_amd", "csrc", f[4])
            if not os.path.exists(src):
                return None
            h = hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]
            if h != f[3]:
                return None
            return {"fetch_bytes": float(f[1]), "write_bytes": float(f[2]), "bytes": float(f[1]) + float(f[2])}
    return None


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1"}))
        sys.exit(2)

    import torch
    from paper_2008_06967_amd import nets, ops, synth

    spec = synth.workload(args.workload)
    xyz_np, feat_np = synth.make_points(spec)
    w = synth.make_weights(spec)
    dev = torch.device("cuda:0")
    xyz = torch.from_numpy(xyz_np).to(dev)
    feat = None if feat_np is None else torch.from_numpy(feat_np).to(dev)
    B = spec["B"]
    print(f"[bench] workload={args.workload} B={B} N={spec['N']} steps={args.steps} warmup={args.warmup}",
          file=sys.stderr, flush=True)

    def time_net(delayed, steps, warmup, graph, inflight=1):
        """Seconds per step.  inflight > 1 keeps that many independent
        batches in flight: each has its own network buffers and graph and
        is replayed on its own stream, round-robin, so one batch's search
        chain overlaps another's MLP chain."""
        nets_ = [nets.build(spec, w, delayed=delayed, device=dev) for _ in range(inflight)]
        streams = [torch.cuda.Stream(device=dev) for _ in range(inflight)]
        runs = []
        for net in nets_:
            if graph:
                g, _ = net.capture(xyz, feat)
                runs.append(g.replay)
            else:
                runs.append(lambda net=net: net.forward(xyz, feat))
        def step(i):
            with torch.cuda.stream(streams[i % inflight]):
                runs[i % inflight]()
        for i in range(warmup):
            step(i)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(steps):
            step(i)
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) / steps

    if args.calibrate_copy:
        # a plain device copy of known size, for scaling FETCH_SIZE/WRITE_SIZE
        src = torch.empty(64 << 20, dtype=torch.float32, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(f"[bench] copy calibration: {src.numel() * 4} bytes read, {dst.numel() * 4} bytes written per copy",
              file=sys.stderr, flush=True)
        del src, dst

    def step_latencies(delayed, steps, warmup, graph):
        """Per-step GPU times of one batch at a time: an event after every
        replay on a backlogged stream; consecutive differences are the
        step times (ms)."""
        net = nets.build(spec, w, delayed=delayed, device=dev)
        stream = torch.cuda.Stream(device=dev)
        run = net.capture(xyz, feat)[0].replay if graph else (lambda: net.forward(xyz, feat))
        with torch.cuda.stream(stream):
            for _ in range(warmup):
                run()
        torch.cuda.synchronize()
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
        with torch.cuda.stream(stream):
            torch.cuda._sleep(int(5e7))
            evs[0].record(stream)
            for i in range(steps):
                run()
                evs[i + 1].record(stream)
        torch.cuda.synchronize()
        t = np.array([evs[i].elapsed_time(evs[i + 1]) for i in range(steps)])
        return {"median": float(np.median(t)), "p10": float(np.percentile(t, 10)), "p90": float(np.percentile(t, 90)),
                "mean": float(t.mean()), "std": float(t.std()), "n": int(steps)}

    graph = not args.eager
    # single-batch latency (one batch at a time)
    t_latency = time_net(True, args.steps, args.warmup, graph, 1)
    lat_stats = step_latencies(True, max(args.steps, 50), args.warmup, graph)
    print(f"[bench] delayed, 1 batch in flight: {t_latency * 1e3:.3f} ms/step", file=sys.stderr, flush=True)
    # throughput with independent batches overlapping
    per_inflight = {1: t_latency}
    for k in (2, 3, 4):
        per_inflight[k] = time_net(True, args.steps, args.warmup, graph, k)
        print(f"[bench] delayed, {k} batches in flight: {per_inflight[k] * 1e3:.3f} ms/step", file=sys.stderr,
              flush=True)
    inflight = min(per_inflight, key=lambda k: per_inflight[k])
    t_step = per_inflight[inflight]
    t_conv_lat = time_net(False, max(5, args.steps // 2), 2, graph, 1)
    t_conv = time_net(False, max(5, args.steps // 2), 2, graph, inflight)
    print(f"[bench] conventional {t_conv_lat * 1e3:.3f} ms/step (1 in flight), {t_conv * 1e3:.3f} ({inflight})",
          file=sys.stderr, flush=True)
    # limited delayed aggregation (Sec. 7.3): fp32 PointNet++ networks
    ltd = None
    if spec["kind"] in ("pointnet2_cls", "pointnet2_seg") and spec.get("dtype") != "bf16":
        t_ltd_lat = time_net("ltd", max(5, args.steps // 2), 2, graph, 1)
        t_ltd = time_net("ltd", max(5, args.steps // 2), 2, graph, inflight)
        print(f"[bench] limited order {t_ltd_lat * 1e3:.3f} ms/step (1 in flight), {t_ltd * 1e3:.3f} ({inflight})",
              file=sys.stderr, flush=True)
        ltd = {"ms_per_step": t_ltd * 1e3, "clouds_per_s": B / t_ltd, "latency_ms_per_batch": t_ltd_lat * 1e3,
               "speedup_vs_conventional": t_conv / t_ltd, "latency_speedup_vs_conventional": t_conv_lat / t_ltd_lat}
    t_step_eager = time_net(True, max(5, args.steps // 2), 2, False, 1)

    # per-call durations (eager pass with events on each call's stream)
    timer = StageTimer(ops)
    timer.install()
    net = nets.build(spec, w, delayed=True, device=dev)
    net.forward(xyz, feat)
    torch.cuda.synchronize()
    timer.active = True
    # hold the streams behind a spin kernel while every call is enqueued, so
    # each event pair brackets GPU execution only (no host launch gaps)
    torch.cuda._sleep(int(2e8))
    for _ in range(max(5, args.steps // 2)):
        timer.begin_step()
        net.forward(xyz, feat)
    stages = timer.summary()
    timer.active = False
    timer.uninstall()

    # dominant kernel = the longest call of the step; roofline for each call
    work = {k: v for k, v in timer.work.items() if v is not None}
    mfma_peak = MFMA_BF16_PEAK_TFLOPS if spec.get("dtype") == "bf16" else MFMA_F32_PEAK_TFLOPS
    roofs = {}
    for k, ms in stages.items():
        if k not in work:
            continue
        kd, am, extra = work[k]
        rate = am / (ms * 1e-3)
        pk, pu = PEAKS[kd]
        if kd == "mfma":
            pk = mfma_peak
        roofs[k] = {"bound": kd, "achieved": round(rate, 4), "peak": pk, "unit": pu, "frac": round(rate / pk, 5)}
        if extra and "logical_gather_bytes" in extra:
            roofs[k]["logical_gather_GBps"] = round(extra["logical_gather_bytes"] / (ms * 1e-3) / 1e9, 1)
        if extra and "serial_iterations" in extra:
            # latency view of a sequential kernel: time per dependent
            # iteration, and the rate against the CUs it can occupy
            roofs[k]["us_per_iteration"] = round(ms * 1e3 / max(1, extra["serial_iterations"]), 4)
            cus = min(extra["workgroups"], N_CUS)
            roofs[k]["frac_of_occupied_cus"] = round(rate / (pk * cus / N_CUS), 5)
        if extra and "compulsory_bytes" in extra:
            gbs = extra["compulsory_bytes"] / (ms * 1e-3) / 1e9
            roofs[k]["hbm_compulsory_GBps"] = round(gbs, 1)
            roofs[k]["hbm_frac"] = round(gbs / HBM_PEAK_GBS, 5)
    dom = max((k for k in stages if k in work), key=lambda k: stages[k])
    roof = dict(roofs[dom])
    roof["kernel"] = dom
    roof["avg_ms"] = stages[dom]
    tr = load_traffic(dom.split("#")[0] + "#" + dom.split("#")[1] + "@" + args.workload)
    roof["traffic"] = None if tr is None else tr["bytes"]

    per_module = {}
    module_ms = {}
    for i, m in enumerate(spec.get("sa", [])):
        per_module[f"sa{i + 1}_centroids_per_s"] = B * m["M"] / t_step
        # serial sum of this module's calls (search + MLP + aggregation)
        ms = sum(stages.get(f"{n}#{i}", 0.0) for n in ("fps", "ball_query", "pointwise_mlp", "aggregate_max"))
        module_ms[f"sa{i + 1}"] = round(ms, 5)
        per_module[f"sa{i + 1}_centroids_per_s_serial_stage_sum"] = B * m["M"] / (ms * 1e-3)

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(spec, xyz_np, feat_np, w, args.cpu_seconds)

    res = {
        "metric": METRIC,
        "value": B / t_step,
        "unit": "clouds/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": t_step * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if spec.get("dtype") != "bf16" else "bf16",
        "data": "synthetic",
        "config": {"workload": f"{args.workload} ({DESCRIBE.get(args.workload, args.workload)}, delayed aggregation)",
                   "global_batch": B, "points": spec["N"], "path": "delayed",
                   "timing": ("eager launches" if args.eager else "HIP graph replay, search chain on a side stream")
                   + f", {inflight} independent batch(es) in flight on separate streams",
                   "batches_in_flight": inflight, "parallelism": "single GPU"},
        "latency_ms_per_batch": t_latency * 1e3,
        "latency_ms_per_batch_stats": {k: (round(v, 5) if isinstance(v, float) else v) for k, v in lat_stats.items()},
        "module_serial_ms": module_ms,
        "clouds_per_s_by_batches_in_flight": {str(k): B / v for k, v in per_inflight.items()},
        "centroids_per_s": per_module,
        "conventional": {"ms_per_step": t_conv * 1e3, "clouds_per_s": B / t_conv, "speedup_delayed": t_conv / t_step,
                         "latency_ms_per_batch": t_conv_lat * 1e3,
                         "latency_speedup_delayed": t_conv_lat / t_latency},
        "limited_order": ltd,
        "eager_ms_per_step": t_step_eager * 1e3,
        "stages_ms": {k: round(v, 5) for k, v in stages.items()},
        "stage_roofline": roofs,
        "critical_path_note": "fps/ball_query run on a side stream concurrently with the MLP chain",
        "roofline": roof,
        "cpu_baseline": cpu,
        "paper_context": {"software_speedup_mobile_gpu": 1.6, "limited_order_speedup_mobile_gpu": 1.3,
                          "hardware_speedup_up_to": 3.6},
    }
    print(json.dumps(res))


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _oracle_rate(spec, xyz, feat, w, seconds, delayed, threads):
    """Clouds/s of the CPU oracle forward over clouds of the batch, one cloud
    per call, on `threads` threads (the oracle's C routines run without the
    interpreter lock), for about `seconds`."""
    import threading
    import oracle.nets as ON
    B = spec["B"]
    lock = threading.Lock()
    state = {"next": 0, "done": 0}
    t0 = time.perf_counter()

    def worker():
        while time.perf_counter() - t0 < seconds:
            with lock:
                c = state["next"] % B
                state["next"] += 1
            sub = dict(spec, B=1)
            ON.forward(sub, xyz[c:c + 1], None if feat is None else feat[c:c + 1], w, delayed=delayed)
            with lock:
                state["done"] += 1

    ts = [threading.Thread(target=worker) for _ in range(threads)]
    for t in ts:
        t.start()
    for t in ts:
        t.join()
    dt = time.perf_counter() - t0
    return state["done"] / dt, state["done"], dt


def cpu_baseline(spec, xyz, feat, w, seconds):
    """The CPU oracle on the same workload: the delayed forward on one
    thread (the reported value), on one thread per available core (up to
    16), and the conventional forward on one thread."""
    cores = min(16, len(os.sched_getaffinity(0)))
    v1, n1, d1 = _oracle_rate(spec, xyz, feat, w, 0.5 * seconds, True, 1)
    vm, nm, dm = _oracle_rate(spec, xyz, feat, w, 0.25 * seconds, True, cores)
    vc, nc, dc = _oracle_rate(spec, xyz, feat, w, 0.25 * seconds, False, 1)
    return {"value": v1, "unit": "clouds/s", "cores": 1, "kind": "oracle",
            "sample": f"{n1} clouds of the batch (delayed forward, fp64 accumulation), {d1:.1f} s, single thread",
            "multithread": {"value": vm, "cores": cores, "sample": f"{nm} clouds in {dm:.1f} s"},
            "conventional_single_thread": {"value": vc, "sample": f"{nc} clouds in {dc:.1f} s"},
            "cpu_model": _cpu_model()}


if __name__ == "__main__":
    main()

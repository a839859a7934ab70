"""Benchmark: PointNet++ SSG segmentation forward of indoor rooms, batch
16 x 4096 points (xyz + 3 features), fp32, delayed aggregation, on one
MI355X -- the largest fp32 workload -- plus every other synthetic workload
under `workloads`.

One step = one full forward of one batch (FPS, ball query, per-point MLP
and aggregation for the four set-abstraction levels, 3-NN interpolation
and feature propagation for the four FP levels, per-point head).  Inputs
and weights are resident in HBM before timing; the timed steps replay a
HIP graph of the two-stream forward (search chain on a side stream), one
batch at a time: `value` = batch / seconds per step, `ms_per_step` = the
batch latency.
The JSON line also carries:
  - conventional / limited_order: the same network in the original order
    (Eq. (1)) and with only the first layer's product hoisted (Sec. 7.3),
    timed with the same steps and warmup, and the latency speedups;
  - throughput_batches_in_flight: independent batches overlapped on
    separate streams (a serving view; not the value);
  - stages: per-call durations from HIP events on the stream each kernel
    runs on (an eager pass), each call's algorithmic work derived from its
    arguments (ball query: the pairs the search rule scans, from its
    output);
  - roofline: the dominant (longest) kernel's achieved rate against MI355X
    peak; `workloads`: the same summary for every workload, with each
    aggregation's HBM fraction and each MLP's MFMA fraction against its
    attainable roof;
  - cpu_baseline: the CPU oracle timed on this host's cores.
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
WORKLOAD = "pointnet2_seg"
ALL_WORKLOADS = "sa_module,pointnet2_cls,dgcnn,pointnet2_seg,pointnet2_seg:bf16,lidar"
DESCRIBE = {
    "sa_module": "one set-abstraction module, 1024 uniform points -> 512 centroids, r 0.2, K 32, 3 -> 64 -> 64 -> 128",
    "pointnet2_cls": "PointNet++ SSG classifier, 1024-point surface clouds, 2 SA levels, group-all, FC head",
    "dgcnn": "DGCNN, 1024-point surface clouds, 4 EdgeConv layers with k = 20 in feature space, "
             "1x1 conv to 1024, global max",
    "pointnet2_seg": "PointNet++ SSG segmentation of 4096-point indoor rooms (xyz + 3 features), "
                     "4 SA levels, 4 FP levels, 13-class head",
    "lidar": "3-level PointNet++ backbone on 16384-point LiDAR sweeps, bf16 MLPs",
}
AGG_TARGET = 0.60    # aggregation: fraction of HBM peak
MLP_TARGET = 0.50    # per-point MLP: fraction of MFMA peak
HBM_PEAK_GBS = 8000.0
MFMA_F32_PEAK_TFLOPS = 157.3
MFMA_BF16_PEAK_TFLOPS = 2516.6
N_CUS = 256   # MI355X compute units (the ALU peak is spread evenly over them)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=WORKLOAD, help="the headline workload (name or name:bf16)")
    ap.add_argument("--workloads", default=ALL_WORKLOADS,
                    help="comma-separated workloads summarised under `workloads` ('' for none)")
    ap.add_argument("--inflight", type=int, default=3, help="most independent batches in flight (secondary view)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
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

    NAMES = ("fps", "fps_prefix", "fps_prefix_levels", "ball_query", "ball_query_grid_build", "ball_query_grid", "knn", "pointwise_mlp", "aggregate_max", "conventional_module", "interpolate3",
             "three_nn", "interpolate3_apply", "interpolate3_add", "interpolate3_mlp", "aggregate_mlp")

    def __init__(self, ops):
        import torch
        self.torch = torch
        self.ops = ops
        self.orig = {n: getattr(ops, n) for n in self.NAMES}
        self.records = []     # (name#k, start, end)
        self.calls = {}       # name#k -> (args, kwargs, result) of the last step
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
                self.calls[f"{__n}#{k}"] = (a, kw, r)
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

    def work(self):
        """name#k -> (bound, amount, extra), after summary() (the ball
        query's work is read from its output)."""
        return {k: w for k, (a, kw, r) in self.calls.items() if (w := call_work(k.split("#")[0], a, kw, r))}


# ----------------------------------------------------------------------------
# algorithmic work of one call, from its arguments (documented in the design doc)
# ----------------------------------------------------------------------------

def call_work(name, a, kw, result=None):
    """(bound, amount, extra) for one entry-point call; amount in TFLOP
    (alu / mfma) or GB (hbm).

    fps:            (M-1) * N point updates per cloud, 8 flops each (3 sub,
                    1 mul, 2 fma) -> alu
    fps_prefix, fps_prefix_levels: the nested sampling as a prefix:
                    compulsory HBM bytes (indices and coordinates read and
                    written) -> hbm
    ball_query_grid_build: the cloud read, its binned copy written -> hbm
    ball_query:     the candidate pairs the search rule scans, 8 flops each
                    -> alu: a query that fills its K slots scans up to its
                    K-th hit (index nit[K-1] + 1), otherwise all N points;
                    read from the call's output (a full list ascends, so
                    nit[K-1] > nit[0]; a short one is padded with nit[0]).
                    B * M * N is reported beside it as the worst case, and
                    the compulsory HBM bytes (points, centroids, NIT)
    knn:            B * M * N pairs, 3 * C flops each (sub, mul, add) -> alu;
                    compulsory bytes (reference and query rows, NIT) beside it
    pointwise_mlp:  2 * rows * sum(C_l * C_l+1) -> mfma
    aggregate_max:  compulsory HBM bytes -- every PFT row read once, the NIT,
                    the centroid indices or rows, the output -> hbm (the
                    bytes of the gathered rows are reported beside it)
    conventional:   2 * B*M*K * sum(C_l * C_l+1) -> mfma
    interpolate3, three_nn: B * Nd * Ns pairs, 8 flops each -> alu
    interpolate3_apply: compulsory HBM bytes (source rows once, neighbours
                    and distances, output) -> hbm
    interpolate3_add: the same plus the added rows -> hbm
    interpolate3_mlp: the MLP's flops on the interpolated rows -> mfma
    """
    def arg(i, key, default=None):
        return a[i] if len(a) > i else kw.get(key, default)

    if name == "fps":
        xyz, M = arg(0, "xyz"), arg(1, "M")
        B, N = xyz.shape[0], xyz.shape[1]
        # one workgroup per cloud walks M - 1 dependent iterations
        return ("alu", 8.0 * B * (M - 1) * N / 1e12, {"serial_iterations": M - 1, "workgroups": B})
    if name == "fps_prefix":
        ip, M = arg(0, "idx_prev"), arg(2, "M")
        return ("hbm", 32.0 * ip.shape[0] * M / 1e9, None)
    if name == "fps_prefix_levels":
        i0, Ms = arg(0, "idx0"), arg(2, "Ms")
        return ("hbm", 32.0 * i0.shape[0] * sum(Ms) / 1e9, None)
    if name == "ball_query_grid_build":
        xyz = arg(0, "xyz")
        return ("hbm", 28.0 * xyz.shape[0] * xyz.shape[1] / 1e9, None)
    if name in ("ball_query", "ball_query_grid"):
        xyz, q, K = arg(0, "xyz"), arg(1, "qxyz"), arg(3, "K")
        B, N, M = xyz.shape[0], xyz.shape[1], q.shape[1]
        comp = 12 * B * N + 12 * B * M + 4 * B * M * K
        nit = result[0] if result is not None else kw.get("out")
        scanned = B * M * N
        if nit is not None and K >= 2:
            full = nit[..., K - 1] > nit[..., 0]
            scanned = int(torch_where_sum(full, nit[..., K - 1].long() + 1, N))
        return ("alu", 8.0 * scanned / 1e12, {"compulsory_bytes": comp, "scanned_pairs": scanned,
                                              "worst_case_pairs": B * M * N})
    if name == "knn":
        ref, q, K = arg(0, "ref"), arg(1, "query"), arg(2, "K")
        B, N, C = ref.shape
        M = q.shape[1]
        comp = 4 * B * N * C + (0 if q.data_ptr() == ref.data_ptr() else 4 * B * M * C) + 4 * B * M * K
        return ("alu", 3.0 * C * B * M * N / 1e12, {"compulsory_bytes": comp})
    if name == "pointwise_mlp":
        x0, prm, x1 = arg(0, "x0"), arg(1, "p"), arg(2, "x1")
        rows = int(np.prod(x0.shape[:-1]))
        d = prm.dims
        out = result if result is not None else kw.get("out")
        wsz = 2 if prm.dtype == 1 else 4
        # a fused MLP's compulsory bytes: its input rows, its output, the weights
        byts = rows * x0.shape[-1] * x0.element_size() + sum(x * y for x, y in zip(d[:-1], d[1:])) * wsz
        if x1 is not None:
            byts += rows * x1.shape[-1] * x1.element_size()
        if out is not None:
            byts += out.numel() * out.element_size()
        return ("mfma", 2.0 * rows * sum(x * y for x, y in zip(d[:-1], d[1:])) / 1e12,
                {"compulsory_bytes_mlp": byts, "bf16": prm.dtype == 1})
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
    if name == "aggregate_mlp":
        # the MLP's flops (its aggregation's bytes beside it)
        pft, nit, prm = arg(1, "pft"), arg(2, "nit"), arg(4, "p")
        B, N, C = pft.shape
        M, K = nit.shape[1], nit.shape[2]
        d = prm.dims
        return ("mfma", 2.0 * B * M * sum(x * y for x, y in zip(d[:-1], d[1:])) / 1e12,
                {"bf16": False, "aggregation_compulsory_bytes": 4 * B * N * C + 4 * B * M * K + 4 * B * M * C})
    if name == "interpolate3_mlp":
        nit, prm = arg(0, "nit"), arg(4, "p")
        rows = nit.shape[0] * nit.shape[1]
        d = prm.dims
        return ("mfma", 2.0 * rows * sum(x * y for x, y in zip(d[:-1], d[1:])) / 1e12, {"bf16": False})
    if name == "conventional_module":
        nit, prm = arg(0, "nit"), arg(1, "p")
        rows = int(np.prod(nit.shape))
        d = prm.dims
        return ("mfma", 2.0 * rows * sum(x * y for x, y in zip(d[:-1], d[1:])) / 1e12, None)
    if name in ("interpolate3", "three_nn"):
        dst, src = arg(0, "xyz_dst"), arg(1, "xyz_src")
        return ("alu", 8.0 * dst.shape[0] * dst.shape[1] * src.shape[1] / 1e12, None)
    if name in ("interpolate3_apply", "interpolate3_add"):
        nit, f = arg(0, "nit"), arg(2, "f_src")
        B, Nd = nit.shape[0], nit.shape[1]
        Ns, C = f.shape[1], f.shape[-1]
        # every source row once, the neighbours and distances, the output
        # (and the added rows)
        comp = 4 * B * Ns * C + 24 * B * Nd + 4 * B * Nd * C
        if name == "interpolate3_add":
            comp += 4 * B * Nd * C
        return ("hbm", comp / 1e9, {"logical_gather_bytes": 12 * B * Nd * C})
    return None


def torch_where_sum(cond, a, b):
    import torch
    return torch.where(cond, a, torch.full_like(a, b)).sum().item()


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


def _spec(tag):
    """'name' or 'name:bf16' -> (spec, label)."""
    from paper_2008_06967_amd import synth
    name, _, dt = tag.partition(":")
    spec = synth.workload(name, **({"dtype": dt} if dt else {}))
    return spec, tag


def measure(tag, args, dev, headline=False):
    """Time one workload: the delayed forward (one batch at a time, graph
    replay), the conventional and limited orders with the same steps and
    warmup, per-call events and rooflines.  Returns (summary, details)."""
    import torch
    from paper_2008_06967_amd import nets, ops, synth

    spec, label = _spec(tag)
    xyz_np, feat_np = synth.make_points(spec)
    w = synth.make_weights(spec)
    xyz = torch.from_numpy(xyz_np).to(dev)
    feat = None if feat_np is None else torch.from_numpy(feat_np).to(dev)
    B = spec["B"]
    graph = not args.eager
    K, W = args.steps, args.warmup
    bf16 = spec.get("dtype") == "bf16"
    print(f"[bench] {label}: B={B} N={spec['N']} dtype={'bf16' if bf16 else 'f32'} steps={K} warmup={W}",
          file=sys.stderr, flush=True)

    def time_net(delayed, inflight=1):
        """Seconds per step over exactly K timed steps after W warmup steps
        (synchronised on both sides).  inflight > 1 keeps that many
        independent batches in flight, each with its own buffers and graph
        on its own stream, replayed round-robin."""
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
        for i in range(W):
            step(i)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(K):
            step(i)
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) / K

    def step_latencies(delayed, steps):
        """Per-step GPU times of one batch at a time: an event after every
        replay on a backlogged stream; consecutive differences are the
        step times (ms)."""
        net = nets.build(spec, w, delayed=delayed, device=dev)
        stream = torch.cuda.Stream(device=dev)
        run = net.capture(xyz, feat)[0].replay if graph else (lambda: net.forward(xyz, feat))
        with torch.cuda.stream(stream):
            for _ in range(W):
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

    t_step = time_net(True)
    lat = step_latencies(True, max(K, 50))
    print(f"[bench] {label} delayed: {t_step * 1e3:.3f} ms/step (one batch in flight)", file=sys.stderr, flush=True)
    t_conv = time_net(False)
    print(f"[bench] {label} conventional: {t_conv * 1e3:.3f} ms/step", file=sys.stderr, flush=True)
    ltd = None
    if spec["kind"] in ("pointnet2_cls", "pointnet2_seg") and not bf16:
        t_ltd = time_net("ltd")
        print(f"[bench] {label} limited order: {t_ltd * 1e3:.3f} ms/step", file=sys.stderr, flush=True)
        ltd = {"ms_per_step": t_ltd * 1e3, "clouds_per_s": B / t_ltd, "speedup_vs_conventional": t_conv / t_ltd,
               "delayed_speedup_vs_limited": t_ltd / t_step}
    inflight = None
    if headline and args.inflight > 1:
        inflight = {"1": B / t_step}
        for k in range(2, args.inflight + 1):
            tk = time_net(True, k)
            inflight[str(k)] = B / tk
            print(f"[bench] {label} delayed, {k} batches in flight: {tk * 1e3:.3f} ms/step", file=sys.stderr,
                  flush=True)

    # per-call durations (eager pass, events on each call's stream)
    timer = StageTimer(ops)
    timer.install()
    net = nets.build(spec, w, delayed=True, device=dev)
    net.forward(xyz, feat)
    torch.cuda.synchronize()
    timer.active = True
    # hold the streams behind a spin kernel while every call is enqueued, so
    # each event pair brackets GPU execution only (no host launch gaps)
    torch.cuda._sleep(int(2e8))
    for _ in range(max(5, min(K, 20))):
        timer.begin_step()
        net.forward(xyz, feat)
    stages = timer.summary()
    timer.active = False
    timer.uninstall()
    work = timer.work()

    mfma_peak = MFMA_BF16_PEAK_TFLOPS if bf16 else MFMA_F32_PEAK_TFLOPS
    roofs = {}
    for k, ms in stages.items():
        if k not in work:
            continue
        kd, am, extra = work[k]
        rate = am / (ms * 1e-3)
        pk, pu = PEAKS[kd]
        if kd == "mfma":
            # each MLP against the peak of the type it computes in
            pk = mfma_peak if not extra or "bf16" not in extra else (
                MFMA_BF16_PEAK_TFLOPS if extra["bf16"] else MFMA_F32_PEAK_TFLOPS)
        r = {"bound": kd, "achieved": round(rate, 4), "peak": pk, "unit": pu, "frac": round(rate / pk, 5),
             "avg_ms": round(ms, 5)}
        extra = extra or {}
        if "logical_gather_bytes" in extra:
            r["logical_gather_GBps"] = round(extra["logical_gather_bytes"] / (ms * 1e-3) / 1e9, 1)
        if "serial_iterations" in extra:
            # latency view of a sequential kernel: time per dependent
            # iteration, and the rate against the CUs it can occupy
            r["us_per_iteration"] = round(ms * 1e3 / max(1, extra["serial_iterations"]), 4)
            cus = min(extra.get("workgroups", N_CUS), N_CUS)
            r["frac_of_occupied_cus"] = round(rate / (pk * cus / N_CUS), 5)
        if "compulsory_bytes" in extra:
            gbs = extra["compulsory_bytes"] / (ms * 1e-3) / 1e9
            r["hbm_compulsory_GBps"] = round(gbs, 1)
            r["hbm_frac"] = round(gbs / HBM_PEAK_GBS, 5)
        if "scanned_pairs" in extra:
            r["scanned_pairs"] = extra["scanned_pairs"]
            r["worst_case_frac"] = round(8.0 * extra["worst_case_pairs"] / 1e12 / (ms * 1e-3) / pk, 5)
        if "compulsory_bytes_mlp" in extra:
            # the roof this MLP can reach: MFMA peak, or HBM peak x its
            # arithmetic intensity when that is lower
            ai = am * 1e12 / extra["compulsory_bytes_mlp"]
            att = min(1.0, ai * HBM_PEAK_GBS * 1e9 / (pk * 1e12))
            r["arithmetic_intensity"] = round(ai, 1)
            r["attainable_frac"] = round(att, 4)
            r["frac_of_attainable"] = round(rate / pk / att, 4)
        roofs[k] = r
    dom = max((k for k in stages if k in work), key=lambda k: stages[k])
    roof = dict(roofs[dom])
    roof["kernel"] = dom
    tr = load_traffic(dom + "@" + label)
    roof["traffic"] = None if tr is None else tr["bytes"]

    per_module, module_ms = {}, {}
    for i, m in enumerate(spec.get("sa", [])):
        per_module[f"sa{i + 1}"] = B * m["M"] / t_step
        ms = sum(stages.get(f"{n}#{i}", 0.0) for n in ("fps", "pointwise_mlp", "aggregate_max"))
        ms += stages.get(f"fps_prefix#{i - 1}", 0.0) if i else 0.0
        # the first level's ball query may run against a prebuilt grid
        grid = "ball_query_grid#0" in stages
        ms += stages.get("ball_query_grid#0", 0.0) if (grid and i == 0) else \
            stages.get(f"ball_query#{i - 1 if grid else i}", 0.0)
        module_ms[f"sa{i + 1}"] = round(ms, 5)
    if spec["kind"] == "dgcnn":
        for l in range(len(spec["edge"])):
            per_module[f"edgeconv{l + 1}"] = B * spec["N"] / t_step

    aggs = {k: {"frac": v["frac"], "meets_target": v["frac"] >= AGG_TARGET} for k, v in roofs.items()
            if k.startswith("aggregate_max")}
    # the MLP target applies to the roof each MLP can reach (MFMA peak, or
    # HBM x its arithmetic intensity when lower)
    mlps = {k: {"frac": v["frac"], "attainable_frac": v["attainable_frac"],
                "meets_target": v["frac"] >= MLP_TARGET * v["attainable_frac"]}
            for k, v in roofs.items() if k.startswith("pointwise_mlp") and "attainable_frac" in v}
    summary = {
        "config": DESCRIBE.get(spec["name"], spec["name"]) + (" (bf16 MLPs)" if bf16 and spec["name"] != "lidar"
                                                              else ""),
        "batch": B, "points": spec["N"], "dtype": "bf16" if bf16 else "f32",
        "ms_per_step": t_step * 1e3, "clouds_per_s": B / t_step,
        "latency_ms_stats": {k: (round(v, 5) if isinstance(v, float) else v) for k, v in lat.items()},
        "centroids_per_s": per_module,
        "module_serial_ms": module_ms,
        "conventional_ms_per_step": t_conv * 1e3,
        "speedup_vs_conventional": t_conv / t_step,
        "limited_order": ltd,
        "dominant_kernel": roof,
        "aggregation_hbm_frac": aggs,
        "mlp_mfma_frac": mlps,
        "stages_ms": {k: round(v, 4) for k, v in stages.items()},
    }
    details = {"stages_ms": {k: round(v, 5) for k, v in stages.items()}, "stage_roofline": roofs,
               "throughput_batches_in_flight": inflight, "spec": spec, "data": (xyz_np, feat_np, w)}
    return summary, details


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1 (multi-GPU sharding is "
                                   "designed, not built)"}))
        sys.exit(2)

    import torch

    dev = torch.device("cuda:0")
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

    head, det = measure(args.workload, args, dev, headline=True)
    workloads = {args.workload: head}
    for tag in [t for t in args.workloads.split(",") if t and t != args.workload]:
        workloads[tag], _ = measure(tag, args, dev)

    spec = det["spec"]
    B = spec["B"]
    cpu = None
    if not args.no_cpu_baseline:
        xyz_np, feat_np, w = det["data"]
        cpu = cpu_baseline(spec, xyz_np, feat_np, w, args.cpu_seconds)

    t_step = head["ms_per_step"] * 1e-3
    res = {
        "metric": METRIC,
        "value": B / t_step,
        "unit": "clouds/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": head["dtype"],
        "data": "synthetic",
        "config": {"workload": f"{args.workload}: {head['config']}, delayed aggregation",
                   "global_batch": B, "points": spec["N"], "path": "delayed",
                   "timing": ("eager launches" if args.eager else "HIP graph replay, search chain on a side stream")
                   + ", one batch at a time", "parallelism": "single GPU"},
        "latency_ms_per_batch_stats": head["latency_ms_stats"],
        "centroids_per_s": head["centroids_per_s"],
        "module_serial_ms": head["module_serial_ms"],
        "conventional": {"ms_per_step": head["conventional_ms_per_step"],
                         "clouds_per_s": B / (head["conventional_ms_per_step"] * 1e-3),
                         "speedup_delayed": head["speedup_vs_conventional"]},
        "limited_order": head["limited_order"],
        "throughput_batches_in_flight": det["throughput_batches_in_flight"],
        "stages_ms": det["stages_ms"],
        "stage_roofline": det["stage_roofline"],
        "roofline": head["dominant_kernel"],
        "workloads": workloads,
        "cpu_baseline": cpu,
        "paper_context": {"software_speedup_mobile_gpu": 1.6, "limited_order_speedup_mobile_gpu": 1.3,
                          "hardware_speedup_up_to": 3.6},
    }
    print(json.dumps(res))


def _cpu_model():
    """model name plus family / model / stepping numbers (some hosts report
    only a generic name)."""
    got = {}
    try:
        for line in open("/proc/cpuinfo"):
            k, _, v = line.partition(":")
            k = k.strip()
            if k in ("model name", "cpu family", "model", "stepping") and k not in got:
                got[k] = v.strip()
            if len(got) == 4:
                break
    except OSError:
        pass
    if not got:
        return "unknown"
    return f"{got.get('model name', '?')} (family {got.get('cpu family', '?')}, model {got.get('model', '?')}, " \
           f"stepping {got.get('stepping', '?')})"


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


def cpu_threads():
    """Threads for the multithreaded oracle leg: every core this process may
    run on, capped by the host's per-job CPU share when one is set
    (OMP_NUM_THREADS)."""
    avail = len(os.sched_getaffinity(0))
    share = os.environ.get("OMP_NUM_THREADS", "")
    return (min(avail, int(share)) if share.isdigit() and int(share) > 0 else avail), avail


def cpu_baseline(spec, xyz, feat, w, seconds):
    """The CPU oracle on the same workload, one cloud per call: the delayed
    forward on every usable core (the reported value; clouds are
    independent), on one thread, and the conventional forward on every
    usable core, each for a bounded share of `seconds`."""
    cores, avail = cpu_threads()
    vm, nm, dm = _oracle_rate(spec, xyz, feat, w, 0.4 * seconds, True, cores)
    v1, n1, d1 = _oracle_rate(spec, xyz, feat, w, 0.3 * seconds, True, 1)
    vc, nc, dc = _oracle_rate(spec, xyz, feat, w, 0.3 * seconds, False, cores)
    return {"value": vm, "unit": "clouds/s", "cores": cores, "kind": "oracle",
            "sample": f"{nm} clouds of the batch, delayed forward (scalar C, fp64 accumulation), one cloud per "
                      f"call on {cores} threads, {dm:.1f} s",
            "affinity_cores": avail,
            "single_thread": {"value": v1, "cores": 1, "sample": f"{n1} clouds in {d1:.1f} s"},
            "conventional": {"value": vc, "cores": cores, "sample": f"{nc} clouds in {dc:.1f} s"},
            "cpu_model": _cpu_model()}


if __name__ == "__main__":
    main()

"""End-to-end parity of the five synthetic workloads, delayed and
conventional, against the oracle's compositions (oracle/nets.py).

Index outputs (FPS, ball query, kNN) are bit-exact; features meet the
normwise bars (1e-4 fp32, 2e-2 bf16).  The workload used by bench.py
(PointNet++ classifier, batch 32, delayed) is checked at its full size in
the same launch configuration (two streams, HIP graph replay)."""
import numpy as np
import pytest
import torch

import oracle.nets as ON
from knn_checks import check_knn_near_ties
from paper_2008_06967_amd import nets, synth
from paper_2008_06967_amd._lib import F32, BF16

pytestmark = pytest.mark.gpu


def normwise(g, r):
    g, r = np.asarray(g, np.float64), np.asarray(r, np.float64)
    return float(np.max(np.abs(g - r)) / max(np.max(np.abs(r)), 1e-30))


def run_gpu(spec, xyz, feat, w, delayed, graph=False, **build_kw):
    net = nets.build(spec, w, delayed=delayed, **build_kw)
    tx = torch.from_numpy(xyz).cuda()
    tf = None if feat is None else torch.from_numpy(feat).cuda()
    if graph:
        g, outs = net.capture(tx, tf)
        g.replay()
    else:
        outs = net.forward(tx, tf)
    torch.cuda.synchronize()
    return {k: v.detach().float().cpu().numpy() if v.dtype == torch.bfloat16 else v.detach().cpu().numpy()
            for k, v in outs.items()}


def check_pointnet(spec, got, ref, tol):
    for i, m in enumerate(ref["modules"]):
        assert np.array_equal(got[f"idx{i}"], m["idx"]), f"level {i} FPS"
        assert np.array_equal(got[f"cxyz{i}"], m["cxyz"]), f"level {i} centroids"
        assert np.array_equal(got[f"nit{i}"], m["nit"]), f"level {i} NIT"
        e = normwise(got[f"f{i}"], m["out"])
        assert e <= tol, f"level {i} features {e}"
    for i, f in enumerate(ref.get("fp", [])):
        if f"fp{i}" not in got:
            # the last level fused with the head: its output is not kept
            assert i == len(ref["fp"]) - 1
            continue
        e = normwise(got[f"fp{i}"], f)
        assert e <= tol, f"fp {i}: {e}"
    e = normwise(got["out"], ref["out"])
    assert e <= tol, f"out {e}"


@pytest.mark.parametrize("delayed", [True, False], ids=["delayed", "conventional"])
def test_sa_module_full(gpu, delayed):
    spec = synth.workload("sa_module")
    xyz, feat = synth.make_points(spec)
    w = synth.make_weights(spec)
    ref = ON.forward(spec, xyz, feat, w, delayed=delayed)
    check_pointnet(spec, run_gpu(spec, xyz, feat, w, delayed), ref, 1e-4)


def test_pointnet2_cls_full_batch_graph(gpu):
    """The benchmarked configuration: batch 32, delayed, graph replay."""
    spec = synth.workload("pointnet2_cls")
    xyz, feat = synth.make_points(spec)
    w = synth.make_weights(spec)
    ref = ON.forward(spec, xyz, feat, w, delayed=True)
    check_pointnet(spec, run_gpu(spec, xyz, feat, w, True, graph=True), ref, 1e-4)


def test_pointnet2_cls_conventional_sampled_clouds(gpu):
    """Full batch 32 on the GPU; the oracle recomputes clouds 0 and 31 (the
    clouds of a batch are independent)."""
    spec = synth.workload("pointnet2_cls")
    xyz, feat = synth.make_points(spec)
    w = synth.make_weights(spec)
    got = run_gpu(spec, xyz, feat, w, False)
    sub = dict(spec, B=2)
    pick = [0, 31]
    ref = ON.forward(sub, xyz[pick], None, w, delayed=False)
    got_s = {k: v[pick] for k, v in got.items()}
    check_pointnet(sub, got_s, ref, 1e-4)


@pytest.mark.parametrize("delayed", [True, False], ids=["delayed", "conventional"])
def test_pointnet2_cls_small_batch(gpu, delayed):
    spec = synth.workload("pointnet2_cls", B=3)
    xyz, feat = synth.make_points(spec)
    w = synth.make_weights(spec)
    ref = ON.forward(spec, xyz, feat, w, delayed=delayed)
    check_pointnet(spec, run_gpu(spec, xyz, feat, w, delayed), ref, 1e-4)


@pytest.mark.parametrize("name,B", [("sa_module", 1), ("pointnet2_cls", 3), ("pointnet2_seg", 1)])
def test_limited_order(gpu, name, B):
    """Limited delayed aggregation (Sec. 7.3) end to end against the oracle's
    limited composition, and against the conventional order it equals."""
    spec = synth.workload(name, B=B)
    xyz, feat = synth.make_points(spec)
    w = synth.make_weights(spec)
    ref = ON.forward(spec, xyz, feat, w, delayed="ltd")
    got = run_gpu(spec, xyz, feat, w, "ltd")
    check_pointnet(spec, got, ref, 1e-4)
    conv = ON.forward(spec, xyz, feat, w, delayed=False)
    assert normwise(got["out"], conv["out"]) <= 1e-4


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("delayed", [True, False], ids=["delayed", "conventional"])
def test_pointnet2_seg(gpu, delayed, dtype):
    spec = synth.workload("pointnet2_seg", B=2, dtype=dtype)
    xyz, feat = synth.make_points(spec)
    w = synth.make_weights(spec)
    ref = ON.forward(spec, xyz, feat, w, delayed=delayed)
    check_pointnet(spec, run_gpu(spec, xyz, feat, w, delayed), ref, 1e-4 if dtype == "f32" else 2e-2)


@pytest.mark.parametrize("delayed", [True, False], ids=["delayed", "conventional"])
def test_lidar_bf16(gpu, delayed):
    spec = synth.workload("lidar", B=1)
    xyz, feat = synth.make_points(spec)
    w = synth.make_weights(spec)
    ref = ON.forward(spec, xyz, feat, w, delayed=delayed)
    check_pointnet(spec, run_gpu(spec, xyz, feat, w, delayed), ref, 2e-2)


@pytest.mark.parametrize("delayed,B", [(True, 2), (False, 2), (True, 16)],
                         ids=["delayed", "conventional", "delayed_full_batch"])
def test_dgcnn_teacher_forced(gpu, delayed, B):
    """Each GPU EdgeConv layer consumes the oracle's previous-layer output,
    so its kNN must match the oracle's bit for bit and its features within
    tolerance (free-running, fp rounding differences could flip near-ties
    in later layers' kNN)."""
    spec = synth.workload("dgcnn", B=B)
    xyz, _ = synth.make_points(spec)
    w = synth.make_weights(spec)
    X = xyz
    ec = ON.edgeconv_delayed if delayed else ON.edgeconv_conventional
    for l, (W, b) in enumerate(w["edge"]):
        r = ec(X, spec["k"], W, b)
        one = dict(spec, edge=[W.shape[0]], conv=4)
        wl = {"edge": [(W, b)], "conv": (np.zeros((4, W.shape[0]), np.float32), np.zeros(4, np.float32))}
        net = nets.build(one, wl, delayed=delayed)
        outs = net.forward(torch.from_numpy(np.ascontiguousarray(X)).cuda())
        torch.cuda.synchronize()
        assert np.array_equal(outs["nit0"].cpu().numpy(), r["nit"]), f"layer {l} kNN"
        e = normwise(outs["x0"].cpu().numpy(), r["out"])
        assert e <= 1e-4, f"layer {l}: {e}"
        X = r["out"]


@pytest.mark.parametrize("delayed", [True, False], ids=["delayed", "conventional"])
def test_dgcnn_free_running(gpu, delayed):
    spec = synth.workload("dgcnn", B=2)
    xyz, _ = synth.make_points(spec)
    w = synth.make_weights(spec)
    ref = ON.forward(spec, xyz, None, w, delayed=delayed)
    got = run_gpu(spec, xyz, None, w, delayed)
    check_knn_near_ties(got, ref, spec["k"], "free running")
    e = normwise(got["out"], ref["out"])
    assert e <= 1e-4, e


def _sampled(spec, got, pick):
    return dict(spec, B=len(pick)), {k: v[pick] for k, v in got.items()}


def test_pointnet2_seg_full_batch_graph_sampled_clouds(gpu):
    """Full batch 16 x 4096 under graph replay (the benchmarked launch);
    the oracle recomputes clouds 0 and 15."""
    spec = synth.workload("pointnet2_seg")
    xyz, feat = synth.make_points(spec)
    w = synth.make_weights(spec)
    got = run_gpu(spec, xyz, feat, w, True, graph=True)
    pick = [0, spec["B"] - 1]
    sub, got_s = _sampled(spec, got, pick)
    ref = ON.forward(sub, xyz[pick], feat[pick], w, delayed=True)
    check_pointnet(sub, got_s, ref, 1e-4)


def test_lidar_full_batch_graph_sampled_cloud(gpu):
    """Full batch 4 x 16384 (bf16 MLPs) under graph replay; the oracle
    recomputes the last cloud."""
    spec = synth.workload("lidar")
    xyz, feat = synth.make_points(spec)
    w = synth.make_weights(spec)
    got = run_gpu(spec, xyz, feat, w, True, graph=True)
    pick = [spec["B"] - 1]
    sub, got_s = _sampled(spec, got, pick)
    ref = ON.forward(sub, xyz[pick], None if feat is None else feat[pick], w, delayed=True)
    check_pointnet(sub, got_s, ref, 2e-2)


def test_dgcnn_full_batch_graph_sampled_clouds(gpu):
    """Full batch 16 x 1024 under graph replay; the oracle recomputes clouds
    0 and 15 free-running (layer 1 searches xyz: exact; later layers search
    GPU features, so near-ties may differ in at most 0.1 % of entries, each
    one checked to be a near-tie)."""
    spec = synth.workload("dgcnn")
    xyz, _ = synth.make_points(spec)
    w = synth.make_weights(spec)
    got = run_gpu(spec, xyz, None, w, True, graph=True)
    pick = [0, spec["B"] - 1]
    sub, got_s = _sampled(spec, got, pick)
    ref = ON.forward(sub, xyz[pick], None, w, delayed=True)
    check_knn_near_ties(got_s, ref, spec["k"], "full batch, graph")
    assert normwise(got_s["out"], ref["out"]) <= 1e-4


@pytest.mark.parametrize("delayed", [True, False], ids=["delayed", "conventional"])
def test_fp_first_product_on_coarse_points(gpu, delayed):
    """Every feature-propagation level takes W1a interp(f) as interp(W1a f)
    on the coarse points plus W1b s + b1 (forced at a small batch): the
    oracle's interpolate-then-MLP within 1e-4, and close to the plain
    order."""
    spec = synth.workload("pointnet2_seg", B=2)
    xyz, feat = synth.make_points(spec)
    w = synth.make_weights(spec)
    ref = ON.forward(spec, xyz, feat, w, delayed=delayed)
    got = run_gpu(spec, xyz, feat, w, delayed, fp_coarse_min_rows=0)
    check_pointnet(spec, got, ref, 1e-4)
    plain = run_gpu(spec, xyz, feat, w, delayed, fp_coarse_min_rows=1 << 40)
    for k in ("out", "fp0", "fp3"):
        assert normwise(got[k], plain[k]) <= 1e-5, k


def test_graph_replay_matches_eager(gpu):
    """Replays interleaved with eager work and synchronisations all match
    the eager result bit for bit (no memset nodes, deterministic kernels)."""
    spec = synth.workload("pointnet2_seg", B=2)
    xyz, feat = synth.make_points(spec)
    w = synth.make_weights(spec)
    net = nets.build(spec, w, delayed=True)
    tx, tf = torch.from_numpy(xyz).cuda(), torch.from_numpy(feat).cuda()
    eager = {k: v.clone() for k, v in net.forward(tx, tf).items()}
    g, outs = net.capture(tx, tf)
    for rep in range(4):
        for v in outs.values():
            v.zero_()
        g.replay()
        torch.cuda.synchronize()
        for k in eager:
            assert torch.equal(outs[k], eager[k]), (rep, k)
        net2 = nets.build(spec, w, delayed=False)      # unrelated eager work between replays
        net2.forward(tx, tf)
        torch.cuda.synchronize()


def test_deterministic(gpu):
    spec = synth.workload("dgcnn", B=2)
    xyz, _ = synth.make_points(spec)
    w = synth.make_weights(spec)
    a = run_gpu(spec, xyz, None, w, True)
    b = run_gpu(spec, xyz, None, w, True)
    for k in a:
        assert np.array_equal(a[k], b[k]), k


@pytest.mark.parametrize("name,B", [("pointnet2_seg", 2), ("pointnet2_cls", 3)])
def test_fused_aggregation_changes_nothing(gpu, name, B):
    """Levels whose aggregation runs in the next MLP's loader give the same
    outputs, bit for bit, as the separate aggregation kernel."""
    spec = synth.workload(name, B=B)
    xyz, feat = synth.make_points(spec)
    w = synth.make_weights(spec)
    tx = torch.from_numpy(xyz).cuda()
    tf = None if feat is None else torch.from_numpy(feat).cuda()
    a = nets.build(spec, w, delayed=True, fuse_aggregation=True)
    b = nets.build(spec, w, delayed=True, fuse_aggregation=False)
    oa = {k: v.clone() for k, v in a.forward(tx, tf).items()}
    ob = b.forward(tx, tf)
    torch.cuda.synchronize()
    for k in ob:
        assert torch.equal(oa[k], ob[k]), k


@pytest.mark.parametrize("name,B", [("pointnet2_seg", 2), ("pointnet2_cls", 3), ("lidar", 1)])
def test_fps_prefix_changes_nothing(gpu, name, B):
    """Sampling every level after the first as the previous level's first M
    centroids gives the same outputs, bit for bit, as running the sampling
    kernel on each level (the levels' indices against the oracle are checked
    by the network tests above)."""
    spec = synth.workload(name, B=B)
    xyz, feat = synth.make_points(spec)
    w = synth.make_weights(spec)
    tx = torch.from_numpy(xyz).cuda()
    tf = None if feat is None else torch.from_numpy(feat).cuda()
    a = nets.build(spec, w, delayed=True, fps_prefix=True)
    b = nets.build(spec, w, delayed=True, fps_prefix=False)
    ga, oa = a.capture(tx, tf)
    ga.replay()
    ob = b.forward(tx, tf)
    torch.cuda.synchronize()
    for k in ob:
        assert torch.equal(oa[k], ob[k]), k


def test_fp_last_level_fused_with_head(gpu):
    """The last feature-propagation level's remaining layers and the head in
    one kernel (weights staged in two phases) give the logits of the
    separate calls within fp32 rounding (the head's first layer sums its
    k steps in another order), at the benchmark's full batch."""
    spec = synth.workload("pointnet2_seg")
    xyz, feat = synth.make_points(spec)
    w = synth.make_weights(spec)
    tx = torch.from_numpy(xyz).cuda()
    tf = torch.from_numpy(feat).cuda()
    a = nets.build(spec, w, delayed=True, fuse_head=True)
    b = nets.build(spec, w, delayed=True, fuse_head=False)
    ga, oa = a.capture(tx, tf)
    ga.replay()
    ob = b.forward(tx, tf)
    torch.cuda.synchronize()
    assert "fp3" not in oa and "fp3" in ob
    assert normwise(oa["out"].cpu().numpy(), ob["out"].cpu().numpy()) <= 1e-5
    for k in ob:
        if k not in ("out", "fp3", "logits"):
            assert torch.equal(oa[k], ob[k]), k

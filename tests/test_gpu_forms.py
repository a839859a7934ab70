"""Launch-shape invariance: the kernels pick their form (workgroup shape,
number of workgroups per cloud, LDS or L2 staging, register / streaming /
MFMA kNN, fused or layer-by-layer MLP) from the sizes.  The same values fed
through different forms, by construction, must give identical results
(exact-arithmetic kernels) or agree within rounding (MLP).  Also: the
debug index-range checks read zero on every workload and count planted
out-of-range entries exactly."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2008_06967_amd import nets, ops, synth

pytestmark = pytest.mark.gpu


def g(s):
    return np.random.default_rng(np.random.SeedSequence([200806967, 55, s]))


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def test_fps_one_workgroup_equals_several():
    """20000 distinct points (one workgroup per cloud) and the same points
    followed by 20000 copies of point 0 (40000 points: several workgroups
    per cloud): the copies' running minimum is 0 from the first iteration,
    so they are never selected and both give the same samples."""
    x = g(1).standard_normal((2, 20000, 3)).astype(np.float32)
    xx = np.concatenate([x, np.repeat(x[:, :1], 20000, axis=1)], 1)
    M = 400
    assert ops.fps_workspace_bytes(2, 20000, M) == 0 and ops.fps_workspace_bytes(2, 40000, M) > 0
    i1, c1 = ops.fps(dev(x), M)
    i2, c2 = ops.fps(dev(xx), M)
    assert torch.equal(i1, i2) and torch.equal(c1, c2)
    ri, _ = O.fps(x, M)
    assert np.array_equal(i1.cpu().numpy(), ri)


def test_fps_register_form_equals_lds_form():
    """512 distinct points (registers only) and the same followed by one
    copy of point 0 (513: the coordinates also in LDS): the copy's running
    minimum is 0 from the start, so both give the same samples."""
    x = g(11).standard_normal((3, 512, 3)).astype(np.float32)
    xx = np.concatenate([x, x[:, :1]], 1)
    i1, c1 = ops.fps(dev(x), 300)
    i2, c2 = ops.fps(dev(xx), 300)
    assert torch.equal(i1, i2) and torch.equal(c1, c2)


def test_ball_query_walk_equals_lds_walk():
    """2047 points (the walk through the caches) and the same plus one point
    far away (2048: the cloud copied into LDS first): the far point never
    falls in a ball, and neither form changes the index order."""
    r = g(12)
    x = r.uniform(-1, 1, (2, 2047, 3)).astype(np.float32)
    xx = np.concatenate([x, np.full((2, 1, 3), 50.0, np.float32)], 1)
    q = np.ascontiguousarray(x[:, :300])
    n1, c1 = ops.ball_query(dev(x), dev(q), 0.3, 32, want_cnt=True)
    n2, c2 = ops.ball_query(dev(xx), dev(q), 0.3, 32, want_cnt=True)
    assert torch.equal(n1, n2) and torch.equal(c1, c2)


def test_knn_register_equals_streaming():
    """1000 references (register form) and the same plus 200 references far
    away (1200: streaming form): the far ones never enter the top 20."""
    r = g(2)
    ref = r.standard_normal((2, 1000, 16)).astype(np.float32)
    far = (1e3 + r.standard_normal((2, 200, 16))).astype(np.float32)
    q = np.ascontiguousarray(ref[:, :300])
    n1, d1 = ops.knn(dev(ref), dev(q), 20, want_dist=True)
    n2, d2 = ops.knn(dev(np.concatenate([ref, far], 1)), dev(q), 20, want_dist=True)
    assert torch.equal(n1, n2) and torch.equal(d1, d2)


def test_knn_mfma_equals_register():
    """64 channels (MFMA bounds + exact re-rank) and the same with two zero
    channels appended (66, not a multiple of 8: register form): a zero
    channel adds fma(0, 0, d) = d, so the distances are identical."""
    ref = g(3).standard_normal((2, 1024, 64)).astype(np.float32)
    pad = np.concatenate([ref, np.zeros((2, 1024, 2), np.float32)], -1)
    n1, d1 = ops.knn(dev(ref), dev(ref), 20, want_dist=True)
    n2, d2 = ops.knn(dev(pad), dev(pad), 20, want_dist=True)
    assert torch.equal(n1, n2) and torch.equal(d1, d2)


@pytest.mark.parametrize("dt", [torch.float32, torch.bfloat16])
def test_aggregation_lds_equals_l2(dt):
    """A batch of 32 classifier-shaped clouds (staged in LDS) and each cloud
    alone (batch 1: the L2 form) give identical rows."""
    r = g(4)
    B, N, M, K, C = 32, 1024, 512, 32, 128
    pft = torch.from_numpy(np.maximum(r.standard_normal((B, N, C)), 0).astype(np.float32)).cuda().to(dt)
    nit = torch.from_numpy(r.integers(0, N, (B, M, K)).astype(np.int32)).cuda()
    cidx = torch.from_numpy(r.integers(0, N, (B, M)).astype(np.int32)).cuda()
    full = ops.aggregate_max(pft, nit, cidx=cidx)
    for b in (0, 17, 31):
        one = ops.aggregate_max(pft[b:b + 1].contiguous(), nit[b:b + 1].contiguous(), cidx=cidx[b:b + 1].contiguous())
        assert torch.equal(one[0], full[b]), b


def test_mlp_fused_and_layerwise_agree():
    """A narrow MLP on 20000 rows (fused kernel) and on 40000 rows (layer by
    layer): the first 20000 rows agree within rounding."""
    r = g(5)
    dims = [67, 64, 64, 128]
    Ws = [(r.standard_normal((dims[i + 1], dims[i])) * np.sqrt(2 / dims[i])).astype(np.float32) for i in range(3)]
    bs = [r.uniform(-0.1, 0.1, dims[i + 1]).astype(np.float32) for i in range(3)]
    p = ops.MLPParams(Ws, bs)
    x = torch.from_numpy(r.standard_normal((40000, 67)).astype(np.float32)).cuda()
    assert ops.mlp_workspace_bytes(20000, p) == 0 and ops.mlp_workspace_bytes(40000, p) > 0
    a = ops.pointwise_mlp(x[:20000].contiguous(), p)
    b = ops.pointwise_mlp(x, p)
    assert float((a - b[:20000]).abs().max() / b[:20000].abs().max()) <= 1e-5


@pytest.mark.parametrize("name,B", [("pointnet2_cls", 4), ("dgcnn", 2), ("pointnet2_seg", 2), ("lidar", 1)])
def test_debug_index_checks_read_zero(name, B):
    spec = synth.workload(name, B=B)
    xyz, feat = synth.make_points(spec)
    w = synth.make_weights(spec)
    net = nets.build(spec, w, delayed=True, debug=True)
    net.forward(dev(xyz), None if feat is None else dev(feat))
    assert len(net._range_counts) >= 2
    assert net.index_errors() == {}


def test_count_out_of_range_counts_planted_entries():
    r = g(6)
    idx = r.integers(0, 1000, 100003).astype(np.int32)
    bad = r.choice(idx.size, 777, replace=False)
    idx[bad[:400]] = -r.integers(1, 50, 400)
    idx[bad[400:]] = 1000 + r.integers(0, 50, 377)
    c = ops.count_out_of_range(dev(idx), 1000)
    assert int(c.item()) == 777
    assert int(ops.count_out_of_range(dev(idx[:0]), 1000).item()) == 0

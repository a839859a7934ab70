"""GPU parity of every C-ABI entry point against the CPU oracle, on seeded
inputs from the shared generators.

Bars: FPS indices, ball-query and kNN neighbor tables, and aggregation of an
identical PFT are bit-exact (values compared as numbers, so +0 == -0);
MLP features are within a normwise relative error of 1e-4 (fp32) or 2e-2
(bf16): max|gpu - oracle| / max|oracle| per output tensor.
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle as O
from paper_2008_06967_amd import ops, synth
from paper_2008_06967_amd._lib import F32, BF16

pytestmark = pytest.mark.gpu

GOLD = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")

TOL = {F32: 1e-4, BF16: 2e-2}


def normwise(g, r):
    g, r = np.asarray(g, np.float64), np.asarray(r, np.float64)
    return float(np.max(np.abs(g - r)) / max(np.max(np.abs(r)), 1e-30))


def dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a)).cuda()
    return t if dtype is None else t.to(dtype)


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def g(stream):
    return synth.rng(77, stream)


# ----------------------------------------------------------------------------
# FPS
# ----------------------------------------------------------------------------

FPS_CASES = [
    ("tiny", 2, 5, 5, "normal"),
    ("one", 3, 1, 1, "normal"),
    ("ragged", 3, 100, 37, "normal"),
    ("grid_ties", 2, 300, 300, "grid"),
    ("n200_one_wave", 3, 200, 180, "normal"),        # 129..256 points: one wave, 4 points per lane
    ("grid_ties_256", 2, 256, 256, "grid"),
    ("dups", 2, 700, 500, "dups"),
    ("sa_module", 1, 1024, 512, "cube"),
    ("cls_sa2", 4, 512, 128, "mesh"),
    ("seg_sa1", 2, 4096, 1024, "normal"),
    ("n2000", 2, 2000, 700, "normal"),
    ("n9000", 1, 9000, 300, "normal"),
    # 513 .. 16384 points: the cloud's coordinates in LDS
    ("lds_smallest_m_eq_n", 3, 513, 513, "normal"),
    ("lds_four_waves_grid", 2, 1000, 1000, "grid"),     # four waves: the block max over four slots
    ("lds_1025_m_eq_n", 3, 1025, 1025, "normal"),
    ("lds_m1", 2, 3000, 1, "normal"),
    ("lds_m65", 2, 2048, 65, "mesh"),                  # one result block plus one
    ("lds_grid_ties", 2, 4096, 1500, "grid"),          # 64 distinct points: ties across waves, zero steps
    ("lds_dups", 1, 8192, 2048, "dups"),
    # 8193 .. 16384 points: spatial order, updates skipped by the box bound
    ("skip_grid_ties", 1, 12000, 700, "grid"),         # equal distances across lanes and waves
    ("skip_ragged", 3, 8193, 300, "normal"),           # one real point in the last thread
    ("skip_m_eq_n", 1, 9000, 9000, "normal"),          # every point, minima down to 0
    ("skip_dups", 1, 16384, 2048, "dups"),             # duplicates: ties inside one thread's slots
    ("skip_same", 1, 10000, 100, "same"),              # one point repeated: every minimum 0 after one step
    ("skip_m33", 2, 16000, 33, "cube"),                # one result block of 32 plus one
    ("skip_m1", 2, 16384, 1, "normal"),
    ("skip_mesh", 2, 16384, 3000, "mesh"),
    ("skip_far_outlier", 1, 12000, 500, "outlier"),    # one point 1e6 away: a coarse grid
    ("lidar_sa1", 1, 16384, 4096, "lidar"),
    ("n20000", 1, 20000, 64, "normal"),
    ("n32768_global_path", 1, 32768, 40, "normal"),   # coordinates re-read from memory per iteration
    ("n_max", 1, 65536, 24, "normal"),                # the documented maximum cloud size
    # more than 32768 points: several single-wave workgroups per cloud that
    # exchange their winners through the workspace
    ("multi_b9_ragged_last_group", 9, 32769, 100, "normal"),   # batch not a multiple of 8; last group 1 point
    ("multi_grid_ties", 2, 40000, 500, "grid"),        # equal distances across groups
    ("multi_dups", 2, 40000, 400, "dups"),            # minima reach 0; re-selection
    ("multi_m2", 4, 33000, 2, "normal"),
    ("multi_m65", 3, 33000, 65, "normal"),             # one result block plus one
    ("multi_n_max", 2, 65536, 300, "normal"),
]


def _points(kind, B, N, r):
    if kind == "grid":
        return r.integers(0, 4, size=(B, N, 3)).astype(np.float32)
    if kind == "dups":
        base = r.standard_normal((B, N // 4, 3)).astype(np.float32)
        return base[:, r.integers(0, N // 4, N)]
    if kind == "cube":
        return synth.uniform_cube(r, B, N)
    if kind == "mesh":
        return synth.mesh_surfaces(r, B, N)
    if kind == "lidar":
        return synth.lidar_scene(r, B, N)
    if kind == "same":
        return np.broadcast_to(r.standard_normal((B, 1, 3)).astype(np.float32), (B, N, 3)).copy()
    if kind == "outlier":
        x = r.standard_normal((B, N, 3)).astype(np.float32)
        x[:, N // 2] = 1e6
        return x
    return r.standard_normal((B, N, 3)).astype(np.float32)


@pytest.mark.parametrize("name,B,N,M,kind", FPS_CASES, ids=[c[0] for c in FPS_CASES])
def test_fps_bit_exact(gpu, name, B, N, M, kind):
    x = _points(kind, B, N, g(1))
    ri, rc = O.fps(x, M)
    need = ops.fps_workspace_bytes(B, N, M)
    # a workspace full of stale bytes: the call clears it itself
    ws = torch.full((max(need, 8),), 0x5A, dtype=torch.uint8, device="cuda")
    idx, cxyz = ops.fps(dev(x), M, ws=ws)
    assert np.array_equal(host(idx), ri)
    assert np.array_equal(host(cxyz), rc)
    if need:
        assert int(ws[:4].view(torch.int32).item()) == 0     # no workgroup gave up waiting


FPS_PREFIX_CASES = [
    # name, B, N, levels (M of each nested sampling), cloud kind
    ("seg_levels", 2, 4096, [1024, 256, 64, 16], "mesh"),
    ("cls_levels", 3, 1024, [512, 128], "mesh"),
    ("lidar_levels", 1, 16384, [4096, 1024, 256], "lidar"),
    ("grid_ties", 2, 3000, [900, 300, 31], "grid"),          # 64 distinct points: zero steps from 64 on
    ("dups", 3, 2000, [700, 699, 1], "dups"),
    ("ragged_b5", 5, 777, [333, 333, 65, 2], "normal"),     # M = M_prev, one result block plus one
]


@pytest.mark.parametrize("name,B,N,levels,kind", FPS_PREFIX_CASES, ids=[c[0] for c in FPS_PREFIX_CASES])
def test_fps_prefix_bit_exact(gpu, name, B, N, levels, kind):
    """The nested sampling equals the oracle's sampling of each level's
    input points, and the sampling kernel's own run on them, bit for bit."""
    x = _points(kind, B, N, g(7))
    idx, cxyz = ops.fps(dev(x), levels[0])
    prev_i, prev_c = idx, cxyz
    zero_steps = False
    for M in levels[1:]:
        pc = host(prev_c)
        ri, rc = O.fps(pc, M)
        i2, c2 = ops.fps_prefix(prev_i, prev_c, M)
        assert np.array_equal(host(i2), ri), (name, M)
        assert np.array_equal(host(c2), rc), (name, M)
        fi, fc = ops.fps(prev_c, M)
        assert torch.equal(fi, i2) and torch.equal(fc, c2)
        zero_steps |= bool((host(i2)[:, 1:] == 0).any())
        prev_i, prev_c = i2, c2
    if kind in ("grid", "dups"):
        assert zero_steps      # the distinct points ran out: steps that take point 0
    # every level at once from the first: the same as the chain, bit for bit
    chain = []
    pi, pc = idx, cxyz
    for M in levels[1:]:
        pi, pc = ops.fps_prefix(pi, pc, M)
        chain.append((pi, pc))
    for (ci, cc), (li, lc) in zip(chain, ops.fps_prefix_levels(idx, cxyz, levels[1:])):
        assert torch.equal(ci, li) and torch.equal(cc, lc)


# ----------------------------------------------------------------------------
# ball query
# ----------------------------------------------------------------------------

BQ_CASES = [
    ("sa_module", 1, 1024, 512, 0.2, 32, "cube"),
    ("cls_sa1", 4, 1024, 512, 0.2, 32, "mesh"),
    ("cls_sa2", 4, 512, 128, 0.4, 64, "mesh"),
    ("ragged", 3, 77, 13, 0.7, 5, "normal"),
    ("k1", 2, 200, 50, 0.5, 1, "normal"),
    ("k100", 2, 300, 40, 1.5, 100, "normal"),
    ("nohit", 1, 50, 10, 1e-3, 8, "normal"),
    ("grid_boundary", 1, 64, 64, 1.0, 16, "grid"),
    ("lidar_sa1", 1, 16384, 4096, 0.1, 64, "lidar"),
    ("k_max", 1, 2000, 24, 3.0, 1024, "normal"),      # the documented maximum K
    # 2048 .. 8191 points: the cloud copied into LDS, 16 queries per workgroup
    ("lds_seg_sa1", 2, 4096, 1024, 0.1, 32, "mesh"),
    ("lds_smallest_ragged_m", 3, 2048, 37, 0.3, 16, "normal"),   # queries not a multiple of 16
    ("lds_k_max", 1, 3000, 20, 3.0, 1024, "normal"),
    ("lds_boundary_ties", 1, 4096, 256, 1.0, 40, "grid"),
    ("lds_dups", 2, 5000, 300, 0.3, 64, "dups"),
    ("lds_largest_nohit", 1, 8191, 64, 1e-4, 8, "normal"),
    # 8192 points and more: the grid form (cells of edge >= r, a hit bitmap
    # per query, the first K set bits)
    ("grid_lidar_sa1", 2, 16384, 4096, 0.1, 64, "lidar"),
    ("grid_uniform", 2, 9000, 700, 0.15, 32, "cube"),
    ("grid_boundary_ties", 1, 8192, 512, 1.0, 40, "grid"),   # integer points: d2 == r2 exactly must not hit
    ("grid_dups", 2, 10000, 300, 0.3, 64, "dups"),
    ("grid_k_max", 1, 8200, 50, 2.0, 1024, "normal"),
    ("grid_nohit", 1, 8192, 64, 1e-4, 8, "normal"),
    ("grid_two_far_clusters", 1, 12000, 400, 0.05, 16, "clusters"),   # 32 cells per axis cap: cells wider than r
    ("grid_queries_outside", 2, 8192, 300, 0.5, 32, "outside"),
    ("grid_n_max", 1, 65536, 256, 0.1, 64, "normal"),
]


@pytest.mark.parametrize("name,B,N,M,r_build,r,K,kind", [
    ("seg_sa1", 2, 4096, 1024, 0.1, 0.1, 32, "mesh"),
    ("lidar_sa1", 1, 16384, 4096, 0.1, 0.1, 64, "lidar"),
    ("ragged_small", 3, 100, 37, 0.5, 0.5, 8, "normal"),
    ("grid_boundary_ties", 1, 2000, 300, 1.0, 1.0, 40, "grid"),
    ("query_radius_above_build", 2, 3000, 200, 0.1, 0.3, 32, "mesh"),   # walks: cells too small
    ("query_radius_below_build", 2, 3000, 200, 0.3, 0.1, 32, "mesh"),
])
def test_ball_query_prebuilt_grid(gpu, name, B, N, M, r_build, r, K, kind):
    """Binning first and querying later gives mesorasi_ball_query's result
    bit for bit (and the oracle's), two queries sharing one grid."""
    x = _points(kind, B, N, g(21))
    q = x[:, g(22).choice(N, M, replace=False)] if M <= N else x
    ref, rcnt, _ = O.ball_query(x, q, r, K)
    grid = ops.ball_query_grid_build(dev(x), r_build)
    for _ in range(2):
        nit, cnt = ops.ball_query_grid(dev(x), dev(q), r, K, grid, want_cnt=True)
        assert np.array_equal(host(nit), ref)
        assert np.array_equal(host(cnt), rcnt)
    nit2, _ = ops.ball_query(dev(x), dev(q), r, K)
    assert torch.equal(nit, nit2)


@pytest.mark.parametrize("name,B,N,M,r,K,kind", BQ_CASES, ids=[c[0] for c in BQ_CASES])
def test_ball_query_bit_exact(gpu, name, B, N, M, r, K, kind):
    rr = g(2)
    if kind == "clusters":     # two tight clusters 100 apart: the grid's cells are far wider than r
        x = np.concatenate([rr.normal(0.0, 0.1, (B, N // 2, 3)), rr.normal(100.0, 0.1, (B, N - N // 2, 3))], 1)
        x = x.astype(np.float32)
    elif kind == "outside":
        x = rr.standard_normal((B, N, 3)).astype(np.float32)
    else:
        x = _points(kind, B, N, rr)
    if kind in ("grid", "normal") and name != "nohit":
        q = x[:, rr.choice(N, M, replace=False)]
    elif name == "nohit":
        q = rr.standard_normal((B, M, 3)).astype(np.float32) + 50.0
    elif kind == "outside":    # queries beyond the cloud's box, some within r of it
        q = x[:, rr.choice(N, M, replace=False)].copy()
        far = q[..., 0] > 1.0
        q[..., 0] = np.where(far, x[..., 0].max(1, keepdims=True) + rr.uniform(0, 0.8, far.shape), q[..., 0])
        q = q.astype(np.float32)
    else:
        _, q = O.fps(x, M)
    rn, rc, _ = O.ball_query(x, q, r, K)
    nit, cnt = ops.ball_query(dev(x), dev(q), r, K, want_cnt=True)
    if ops.ball_query_workspace_bytes(B, N, M):
        # a workspace of stale bytes: the grid is rebuilt by the call
        ws = torch.full((ops.ball_query_workspace_bytes(B, N, M),), 0x7F, dtype=torch.uint8, device="cuda")
        n2, c2 = ops.ball_query(dev(x), dev(q), r, K, want_cnt=True, ws=ws)
        assert torch.equal(n2, nit) and torch.equal(c2, cnt)
    assert np.array_equal(host(nit), rn)
    assert np.array_equal(host(cnt), rc)


# ----------------------------------------------------------------------------
# kNN
# ----------------------------------------------------------------------------

KNN_CASES = [
    ("dgcnn_l1", 2, 1024, 1024, 3, 20, "self"),
    ("dgcnn_l2", 2, 1024, 1024, 64, 20, "self"),
    ("dgcnn_l4", 1, 1024, 1024, 128, 20, "self"),
    ("ragged", 3, 100, 37, 5, 7, "other"),
    ("k1", 2, 70, 70, 3, 1, "self"),
    ("k64", 1, 200, 50, 16, 64, "other"),
    ("ties", 2, 150, 150, 3, 10, "grid"),
    ("ties_4ch_groups", 2, 150, 150, 8, 10, "grid"),      # 16-byte channel path with exact ties
    ("c28_scalar_path", 1, 90, 90, 28, 5, "self"),         # 4-channel groups, bank-conflicting stride: scalar path
    ("interp_like", 2, 256, 1024, 3, 3, "other"),
    ("k_max_c_max", 1, 300, 100, 128, 64, "other"),   # the documented maximum K and width
    # at most 1024 points: all distances in registers, one selection per query;
    # few distinct points put far more than 64 candidates at the threshold
    ("reg_ties_many", 2, 1024, 1024, 2, 20, "grid"),
    ("reg_k64", 1, 1024, 256, 8, 64, "other"),
    ("reg_n65", 2, 65, 65, 4, 20, "self"),
    # C in [32, 128], C % 8 == 0, N <= 1024: Gram distances on MFMA bound the
    # exact ones; candidates re-ranked with the exact fp32 distance
    ("mfma_c32_ties", 1, 512, 512, 32, 20, "grid"),
    ("mfma_c96_ragged", 2, 700, 300, 96, 16, "other"),
    ("mfma_near_duplicates", 1, 1024, 256, 64, 20, "jitter"),   # far more candidates than K in the margin
    ("mfma_large_offset", 1, 1000, 200, 128, 20, "offset"),     # norms >> distances: wide margins
    ("mfma_k64", 1, 1024, 128, 128, 64, "other"),
    # C > 64 with C % 16 == 0: 16 queries per workgroup on 16 x 16 MFMA blocks
    ("mfma16_ties_ragged", 2, 333, 77, 80, 20, "grid"),
    ("mfma16_near_duplicates", 1, 1024, 200, 128, 20, "jitter"),
    ("mfma16_overflow", 1, 512, 64, 128, 20, "huge"),
    ("mfma16_m17", 2, 1024, 17, 112, 8, "other"),        # one full block of 16 queries plus one
    # more than 1024 points: the streaming running list
    ("stream_n1500", 1, 1500, 200, 16, 20, "other"),
    ("stream_ties", 1, 1100, 300, 3, 10, "grid"),
    # coordinates around 1e20: most squared distances overflow to +inf, and the
    # list still fills with the lowest such indices (never an empty slot)
    ("stream_overflow", 1, 1500, 100, 3, 20, "huge"),
    ("reg_overflow", 1, 1000, 100, 3, 20, "huge"),
    ("mfma_overflow", 1, 512, 64, 64, 20, "huge"),
]


@pytest.mark.parametrize("name,B,N,M,C,K,kind", KNN_CASES, ids=[c[0] for c in KNN_CASES])
def test_knn_bit_exact(gpu, name, B, N, M, C, K, kind):
    rr = g(3)
    if kind == "grid":
        ref = rr.integers(0, 3, size=(B, N, C)).astype(np.float32)
    elif kind == "jitter":   # 8 base points, each repeated with 1e-6 noise
        base = rr.standard_normal((B, 8, C))
        ref = np.ascontiguousarray(base[:, rr.integers(0, 8, N)] + 1e-6 * rr.standard_normal((B, N, C)), np.float32)
    elif kind == "offset":   # features around 100: |x|^2 ~ 1e6 C, distances ~ 2C
        ref = (100.0 + rr.standard_normal((B, N, C))).astype(np.float32)
    elif kind == "huge":     # finite inputs whose squared distances mostly overflow
        ref = (1e20 * rr.standard_normal((B, N, C))).astype(np.float32)
    else:
        ref = rr.standard_normal((B, N, C)).astype(np.float32)
    if kind in ("self", "grid", "jitter", "offset", "huge"):
        query = ref if M == N else np.ascontiguousarray(ref[:, :M])
    else:
        query = rr.standard_normal((B, M, C)).astype(np.float32)
    rn, rd = O.knn(ref, query, K)
    if kind == "huge":
        assert np.isinf(rd).mean() > 0.5
    nit, dist = ops.knn(dev(ref), dev(query), K, want_dist=True)
    assert np.array_equal(host(nit), rn)
    assert np.array_equal(host(dist), rd)


def test_knn_strided_columns(gpu):
    """Reference/query as a column slice of a wider buffer (leading dim > C)."""
    rr = g(4)
    wide = rr.standard_normal((2, 300, 40)).astype(np.float32)
    rn, _ = O.knn(wide[:, :, 8:24], wide[:, :, 8:24], 20)
    t = dev(wide)
    nit, _ = ops.knn(t[:, :, 8:24], t[:, :, 8:24], 20)
    assert np.array_equal(host(nit), rn)


# ----------------------------------------------------------------------------
# aggregation (identical PFT on both sides: bit-exact)
# ----------------------------------------------------------------------------

AGG_CASES = [
    ("sa_module", 1, 1024, 512, 32, 128, "f32", "cidx"),
    ("cls_sa2", 2, 512, 128, 64, 256, "f32", "cidx"),
    ("lidar_bf16", 1, 4096, 1024, 64, 128, "bf16", "cidx"),
    ("dgcnn_add_relu", 2, 1024, 1024, 20, 64, "f32", "cfeat"),
    ("dgcnn_bf16", 1, 300, 300, 20, 64, "bf16", "cfeat"),
    ("odd_channels", 2, 100, 33, 7, 13, "f32", "cidx"),
    ("odd_bf16", 2, 100, 33, 7, 13, "bf16", "cidx"),
    ("wide", 1, 64, 16, 32, 1024, "f32", "cidx"),
    ("wide_bf16", 1, 64, 16, 32, 2048, "bf16", "cidx"),
    ("none", 2, 80, 20, 5, 24, "f32", "none"),
    ("k1", 2, 50, 50, 1, 8, "f32", "cidx"),
    # batches large enough for the LDS form (a PFT column slice per workgroup)
    ("lds_cls_sa1", 32, 1024, 512, 32, 128, "f32", "cidx"),
    ("lds_cls_sa2", 32, 512, 128, 64, 256, "f32", "cidx"),
    ("lds_dgcnn", 16, 1024, 1024, 20, 64, "f32", "cfeat"),
    ("lds_bf16", 64, 512, 256, 16, 128, "bf16", "cidx"),
    ("lds_bf16_cfeat", 16, 1024, 1024, 20, 128, "bf16", "cfeat"),
    ("lds_ragged_c", 40, 600, 300, 12, 100, "f32", "cidx"),
]


@pytest.mark.parametrize("name,B,N,M,K,C,dt,cen", AGG_CASES, ids=[c[0] for c in AGG_CASES])
def test_aggregate_bit_exact(gpu, name, B, N, M, K, C, dt, cen):
    rr = g(5)
    pft = (rr.standard_normal((B, N, C)) * 3).astype(np.float32)
    if dt == "bf16":
        pft = O.bf16_round(pft)
    nit = rr.integers(0, N, (B, M, K)).astype(np.int32)
    cidx = rr.integers(0, N, (B, M)).astype(np.int32) if cen == "cidx" else None
    cfeat = O.bf16_round(rr.standard_normal((B, M, C)).astype(np.float32)) if cen == "cfeat" else None
    sign = +1 if cen == "cfeat" else -1
    relu = cen == "cfeat"
    ref = O.aggregate_max(pft, nit, cidx=cidx, cfeat=cfeat, sign=sign, relu=relu)
    tdt = torch.float32 if dt == "f32" else torch.bfloat16
    out = ops.aggregate_max(dev(pft).to(tdt), dev(nit), cidx=None if cidx is None else dev(cidx),
                            cfeat=None if cfeat is None else dev(cfeat).to(tdt), sign=sign, relu=relu)
    assert np.array_equal(host(out), ref)


@pytest.mark.parametrize("B", [2, 16])
def test_aggregate_strided_pft_and_out(gpu, B):
    """DGCNN layout: PFT = [A | Bm] in one [N, 2C] table, output into a
    column slice of a wider concat buffer (B = 16 takes the LDS form)."""
    rr = g(6)
    N, K, C = 200, 20, 64
    P = rr.standard_normal((B, N, 2 * C)).astype(np.float32)
    nit = rr.integers(0, N, (B, N, K)).astype(np.int32)
    ref = O.aggregate_max(np.ascontiguousarray(P[..., C:]), nit, cfeat=np.ascontiguousarray(P[..., :C]), sign=+1,
                          relu=True)
    t = dev(P)
    cat = torch.full((B, N, 5 * C), 7.0, device="cuda")
    ops.aggregate_max(t[..., C:], dev(nit), cfeat=t[..., :C], sign=+1, relu=True, out=cat[..., 2 * C:3 * C])
    c = host(cat)
    assert np.array_equal(c[..., 2 * C:3 * C], ref)
    assert (c[..., :2 * C] == 7.0).all() and (c[..., 3 * C:] == 7.0).all()


# ----------------------------------------------------------------------------
# MLP
# ----------------------------------------------------------------------------

MLP_CASES = [
    ("sa1_f32", 1000, [3], [64, 64, 128], F32),
    ("sa2_two_src", 517, [3, 128], [128, 128, 256], F32),
    ("sa3_groupall", 256, [3, 256], [256, 512, 1024], F32),
    # [x0 | x1] with x0 at most 4 wide and x1 aligned: the k loop over x1,
    # x0 added in the epilogue (with split K when the tiles are few)
    ("two_src_splitk", 100, [3, 256], [512, 64], F32),
    ("two_src_x0_1", 300, [1, 64], [64], F32),
    ("two_src_x0_4", 259, [4, 32], [200, 16], F32),
    ("two_src_x0_5", 130, [5, 32], [48], F32),        # x0 too wide: general loader
    ("fc_head", 32, [1024], [512, 256, 40], F32),
    # at most 64 rows: the skinny path (16-column MFMA blocks, K split over waves)
    ("fc_skinny_1row", 1, [1024], [512, 256, 40], F32),
    ("fc_skinny_17rows", 17, [256], [100, 40], F32),
    ("fc_skinny_64rows", 64, [64], [48, 12], F32),
    ("fc_skinny_long_k", 33, [4096], [36], F32),
    ("fc_skinny_unaligned_widths", 20, [30], [22, 6], F32),   # widths not multiples of 4: GEMM path
    ("seg_head", 300, [128], [128, 13], F32),
    ("odd_widths", 77, [5, 2], [33, 17, 9], F32),
    ("sa1_bf16", 1000, [3], [32, 32, 64], BF16),
    ("sa2_bf16_two_src", 333, [3, 64], [64, 64, 128], BF16),
    ("fp_bf16", 200, [256, 128], [256, 256], BF16),
    ("odd_bf16", 45, [6, 1], [20, 12], BF16),
    ("width_max", 40, [4096], [4096, 64], F32),       # the documented maximum width (skinny path)
    ("width_max_gemm", 200, [4096], [4096, 64], F32), # the same on the tiled GEMM path
    ("depth_max", 100, [16], [32] * 8, F32),          # the documented maximum depth
    # a full wave of 256 x 128 tiles (eight-wave kernel), ragged rows and columns
    ("many_rows_wide", 16284, [64], [1000, 384], F32),
    # eight-wave 128 x 128 and 128 x 64 tiles on the split two-source form and
    # on the general loader (widths not multiples of 4, ragged rows)
    ("split_8wave_128x128", 16384, [3, 128], [256], F32),
    ("split_8wave_128x64", 16384, [3, 128], [128], F32),
    ("general_8wave_128x128", 16383, [6, 125], [256], F32),
    # above 32768 rows with every layer at most 128 wide: the register-resident
    # MLP (persistent workgroups, activations in registers between layers)
    ("rr_two_layers", 65536, [128], [128, 128], F32),
    ("rr_head_ragged", 65537, [128], [128, 13], F32),      # last tile of one row; linear last layer
    ("rr_two_src", 40000, [3, 3], [32, 32, 64], F32),      # element loads of [x0 | x1]
    ("rr_odd_widths", 33001, [5, 2], [33, 17, 9], F32),    # partial 32-channel blocks
    ("rr_depth_max", 32769, [16], [32] * 8, F32),
    # weights beyond the LDS: staged in phases (at most one 32-row tile per wave)
    ("rr_staged_head", 65536, [128], [128, 128, 128, 13], F32),
    ("rr_staged_ragged", 40001, [128], [128, 128, 128, 128, 36], F32),
    ("staged_too_many_rows", 65600, [128], [128, 128, 128, 13], F32),   # beyond one tile per wave: the GEMMs
    ("rr_unaligned_out", 40000, [128], [98], F32),        # 98-float output rows: element stores
    # the bf16 form (v_mfma_f32_32x32x16_bf16, activations packed in
    # registers), used for first layers of at most 32 inputs
    ("rr_bf16_two_src", 65536, [3, 3], [32, 32, 64], BF16),
    ("rr_bf16_wide_ragged", 40001, [32], [128, 128, 13], BF16),
    ("rr_bf16_odd_widths", 33001, [5, 2], [33, 17, 9], BF16),
    ("rr_bf16_depth_max", 32769, [16], [32] * 8, BF16),
]


def _weights(rr, dims):
    Ws = [(rr.standard_normal((dims[i + 1], dims[i])) * np.sqrt(2.0 / dims[i])).astype(np.float32)
          for i in range(len(dims) - 1)]
    bs = [rr.uniform(-0.1, 0.1, dims[i + 1]).astype(np.float32) for i in range(len(dims) - 1)]
    return Ws, bs


@pytest.mark.parametrize("name,rows,srcs,widths,dt", MLP_CASES, ids=[c[0] for c in MLP_CASES])
def test_mlp_parity(gpu, name, rows, srcs, widths, dt):
    rr = g(7)
    xs = [rr.standard_normal((rows, c)).astype(np.float32) for c in srcs]
    dims = [sum(srcs)] + widths
    Ws, bs = _weights(rr, dims)
    relu_mask = (1 << (len(widths) - 1)) - 1 if name.startswith("fc") or "head" in name else (1 << len(widths)) - 1
    ref = O.mlp(np.concatenate(xs, -1), Ws, bs, relu_mask=relu_mask, bf16=dt == BF16)
    p = ops.MLPParams(Ws, bs, dtype=dt)
    y = ops.pointwise_mlp(dev(xs[0]), p, x1=dev(xs[1]) if len(xs) > 1 else None, relu_mask=relu_mask)
    assert normwise(host(y), ref) <= TOL[dt]
    if dt == BF16:   # stored activations are bf16 values
        yb = ops.pointwise_mlp(dev(xs[0]), p, x1=dev(xs[1]) if len(xs) > 1 else None, relu_mask=relu_mask,
                               out_dtype=BF16)
        assert yb.dtype == torch.bfloat16
        assert np.array_equal(host(yb.float()), host(y))


@pytest.mark.parametrize("dt", [F32, BF16])
@pytest.mark.parametrize("G", [128, 20, 64, 1])
def test_mlp_pooled(gpu, dt, G):
    rr = g(8)
    groups = 7
    rows = G * groups
    x = rr.standard_normal((rows, 10)).astype(np.float32)
    Ws, bs = _weights(rr, [10, 48, 80])
    ref = O.rowgroup_max(O.mlp(x, Ws, bs, bf16=dt == BF16).reshape(groups, G, 80), G)
    p = ops.MLPParams(Ws, bs, dtype=dt)
    y = ops.pointwise_mlp(dev(x), p, pool_group=G)
    assert normwise(host(y).reshape(groups, 80), ref.reshape(groups, 80)) <= TOL[dt]


def test_mlp_pooled_many_rows(gpu):
    """Per-point 1x1 convolution with the max over each cloud fused, at a
    row count that fills the chip with 256 x 128 tiles."""
    rr = g(12)
    G, groups = 1024, 16
    x = rr.standard_normal((G * groups, 96)).astype(np.float32)
    Ws, bs = _weights(rr, [96, 1024])
    ref = O.rowgroup_max(O.mlp(x, Ws, bs).reshape(groups, G, 1024), G)
    y = ops.pointwise_mlp(dev(x), ops.MLPParams(Ws, bs), pool_group=G)
    assert normwise(host(y).reshape(groups, 1024), ref.reshape(groups, 1024)) <= 1e-4


@pytest.mark.parametrize("G", [32, 16])
def test_mlp_pooled_two_source(gpu, G):
    """Group-all shape: [xyz | features] with the max over each cloud fused."""
    rr = g(10)
    groups = 9
    rows = G * groups
    x0 = rr.standard_normal((rows, 3)).astype(np.float32)
    x1 = rr.standard_normal((rows, 64)).astype(np.float32)
    Ws, bs = _weights(rr, [67, 256])
    ref = O.rowgroup_max(O.mlp(np.concatenate([x0, x1], -1), Ws, bs).reshape(groups, G, 256), G)
    y = ops.pointwise_mlp(dev(x0), ops.MLPParams(Ws, bs), x1=dev(x1), pool_group=G)
    assert normwise(host(y).reshape(groups, 256), ref.reshape(groups, 256)) <= 1e-4


@pytest.mark.parametrize("rows_per_group,groups", [(16, 9), (40, 5)])
def test_mlp_pooled_multilayer_reuses_output(gpu, rows_per_group, groups):
    """A pooled multi-layer MLP on the tiled GEMM path clears its output in
    the first layer's kernel: a second call into the same buffer with
    smaller activations must not keep the first call's maxima."""
    rr = g(11)
    G = rows_per_group
    rows = G * groups
    Ws, bs = _weights(rr, [20, 200, 300])
    p = ops.MLPParams(Ws, bs)
    y = torch.empty(groups, 300, device="cuda")
    for scale in (10.0, 0.1):
        x = (scale * rr.standard_normal((rows, 20))).astype(np.float32)
        ref = O.rowgroup_max(O.mlp(x, Ws, bs).reshape(groups, G, 300), G)
        ops.pointwise_mlp(dev(x), p, pool_group=G, out=y)
        assert normwise(host(y), ref.reshape(groups, 300)) <= 1e-4


def test_mlp_strided_input(gpu):
    rr = g(9)
    wide = rr.standard_normal((100, 50)).astype(np.float32)
    Ws, bs = _weights(rr, [20, 16])
    ref = O.mlp(wide[:, 10:30], Ws, bs)
    t = dev(wide)
    y = ops.pointwise_mlp(t[:, 10:30], ops.MLPParams(Ws, bs))
    assert normwise(host(y), ref) <= 1e-4


# ----------------------------------------------------------------------------
# conventional module, interpolation, small entry points
# ----------------------------------------------------------------------------

# (B, N, M, K, cf, hidden/output widths, dtype, feature row stride or 0):
# fp32 rows are gathered straight from the inputs -- in the fused kernel
# when every layer is narrow, through a split first layer otherwise -- and
# the neighbor matrix is built only for bf16, for feature widths that are
# not a multiple of 4, and for unaligned feature rows.
CONV_CASES = {
    "fused_gather": (2, 512, 128, 32, 13, [32, 48], F32, 0),
    "fused_xyz_only": (3, 300, 70, 32, 0, [32, 64], F32, 0),
    "fused_k20": (2, 256, 50, 20, 8, [40, 24], F32, 0),
    "split_gather": (2, 256, 64, 32, 128, [128, 256], F32, 0),
    "split_strided_k24": (3, 200, 45, 24, 64, [96, 160], F32, 72),
    "nfm_width": (2, 256, 40, 16, 130, [64, 160], F32, 0),
    "bf16": (2, 512, 128, 32, 13, [32, 48], BF16, 0),
}


@pytest.mark.parametrize("case", list(CONV_CASES), ids=list(CONV_CASES))
def test_conventional_pointnet(gpu, case):
    B, N, M, K, cf, widths, dt, ldf = CONV_CASES[case]
    rr = g(10)
    xyz = synth.mesh_surfaces(rr, B, N)
    base = rr.standard_normal((B, N, max(cf, ldf, 1))).astype(np.float32)
    feat = np.ascontiguousarray(base[:, :, :cf]) if cf else None
    idx, cxyz = O.fps(xyz, M)
    nit, _, _ = O.ball_query(xyz, cxyz, 0.4, K)
    Ws, bs = _weights(rr, [3 + cf] + widths)
    h = O.mlp(O.group_pointnet(xyz, feat, cxyz, nit), Ws, bs, bf16=dt == BF16)
    ref = O.rowgroup_max(h.reshape(B, M * K, widths[-1]), K)
    tf = dev(base)[:, :, :cf] if cf else None   # row stride max(cf, ldf)
    out = ops.conventional_module(dev(nit), ops.MLPParams(Ws, bs, dtype=dt), xyz=dev(xyz), feat=tf,
                                  cxyz=dev(cxyz), grouping=0)
    assert normwise(host(out), ref) <= TOL[dt]


def test_conventional_edge(gpu):
    rr = g(11)
    B, N, K, C = 2, 256, 20, 24
    X = rr.standard_normal((B, N, C)).astype(np.float32)
    nit, _ = O.knn(X, X, K)
    Ws, bs = _weights(rr, [2 * C, 40])
    h = O.mlp(O.group_edge(X, nit), Ws, bs)
    ref = O.rowgroup_max(h.reshape(B, N * K, 40), K)
    out = ops.conventional_module(dev(nit), ops.MLPParams(Ws, bs), feat=dev(X), grouping=1)
    assert normwise(host(out), ref) <= 1e-4


# (C1, remaining widths, bias, dtype, p1 row stride): fp32 first-layer rows
# are formed in the next layer's loader -- the fused kernel when every layer
# is narrow, the gathered GEMM otherwise -- and materialized only for bf16
# and for widths or strides that are not a multiple of 4.
LTD_CASES = {
    "fused_vec4": (64, [24, 40], True, F32, 64),
    "fused_scalar_width": (10, [24, 40], True, F32, 10),
    "fused_no_bias": (64, [24, 40], False, F32, 64),
    "gemm_gather": (128, [128, 256], True, F32, 128),
    "gemm_gather_no_bias_strided": (64, [96, 160], False, F32, 72),
    "gemm_materialized": (66, [64, 200], True, F32, 66),
    "bf16_rest": (32, [24, 40], True, BF16, 32),
    # 16384 gathered rows into 256 columns: the eight-wave 128 x 128 tile
    "gemm_gather_8wave": (128, [256, 64], True, F32, 128, (2, 2048, 512, 16)),
}


@pytest.mark.parametrize("case", list(LTD_CASES), ids=list(LTD_CASES))
def test_ltd_module_parity(gpu, case):
    """Limited delayed aggregation (first-layer rows from p1 - q + b1, then
    the remaining layers and the max over K) against the oracle."""
    C1, widths, bias, dt, ldp, *sizes = LTD_CASES[case]
    rr = g(14)
    B, N, M, K = sizes[0] if sizes else (2, 300, 77, 9)
    base = rr.standard_normal((B, N, ldp)).astype(np.float32)
    p1 = np.ascontiguousarray(base[:, :, :C1])
    q = rr.standard_normal((B, M, C1)).astype(np.float32)
    b1 = rr.uniform(-0.2, 0.2, C1).astype(np.float32) if bias else None
    nit = rr.integers(0, N, size=(B, M, K)).astype(np.int32)
    dims = [C1] + widths
    Ws, bs = _weights(rr, dims)
    h1 = O.ltd_group(p1, q, b1, nit)
    h = O.mlp(h1, Ws, bs, bf16=dt == BF16)
    ref = O.rowgroup_max(h.reshape(B, M * K, dims[-1]), K)
    p = ops.MLPParams(Ws, bs, dtype=dt)
    tp = dev(base)[:, :, :C1]   # row stride ldp
    out = ops.ltd_module(tp, dev(q), dev(nit), p, b1=None if b1 is None else dev(b1))
    assert normwise(host(out), ref) <= TOL[dt]


@pytest.mark.parametrize("B,Nd,Ns,C", [(2, 4096, 1024, 128), (3, 100, 17, 5), (1, 64, 16, 512), (2, 10, 3, 8),
                                       (1, 300, 2500, 7), (2, 129, 3, 4)])
def test_interpolate3(gpu, B, Nd, Ns, C):
    rr = g(12)
    dst = rr.uniform(-1, 1, (B, Nd, 3)).astype(np.float32)
    src = np.concatenate([dst[:, :min(Ns, Nd) // 2], rr.uniform(-1, 1, (B, Ns - min(Ns, Nd) // 2, 3))], 1)
    src = src.astype(np.float32)
    f = rr.standard_normal((B, Ns, C)).astype(np.float32)
    ref = O.interpolate3(dst, src, f)
    out = ops.interpolate3(dev(dst), dev(src), dev(f))
    assert normwise(host(out), ref) <= 1e-5


@pytest.mark.parametrize("Ns_half", [40, 700])
def test_interpolate3_ties_take_lowest_index(gpu, Ns_half):
    """Every source point appears twice (indices i and i + Ns_half) with
    different features: equal distances must resolve to the lower index,
    across source chunks and across the waves that split them."""
    rr = g(13)
    base = rr.uniform(-1, 1, (2, Ns_half, 3)).astype(np.float32)
    src = np.concatenate([base, base], 1)
    dst = rr.uniform(-1, 1, (2, 257, 3)).astype(np.float32)
    f = rr.standard_normal((2, 2 * Ns_half, 6)).astype(np.float32)
    ref = O.interpolate3(dst, src, f)
    out = ops.interpolate3(dev(dst), dev(src), dev(f))
    assert normwise(host(out), ref) <= 1e-5


@pytest.mark.parametrize("B,Nd,Ns,C", [(2, 4096, 1024, 128), (3, 100, 17, 5), (2, 10, 3, 8), (1, 300, 2500, 7),
                                       (16, 64, 16, 512)])
def test_three_nn_and_apply(gpu, B, Nd, Ns, C):
    """The split form: the search is the oracle's 3-NN bit for bit (indices
    and squared distances), and the interpolation from it equals the fused
    kernel's output bit for bit and the oracle's within 1e-5."""
    rr = g(15)
    dst = rr.uniform(-1, 1, (B, Nd, 3)).astype(np.float32)
    src = np.concatenate([dst[:, :min(Ns, Nd) // 2], rr.uniform(-1, 1, (B, Ns - min(Ns, Nd) // 2, 3))], 1)
    src = src.astype(np.float32)
    f = rr.standard_normal((B, Ns, C)).astype(np.float32)
    rn, rd = O.knn(src, dst, 3)
    nit, dist = ops.three_nn(dev(dst), dev(src))
    assert np.array_equal(host(nit), rn)
    assert np.array_equal(host(dist), rd)
    out = ops.interpolate3_apply(nit, dist, dev(f))
    fused = ops.interpolate3(dev(dst), dev(src), dev(f))
    assert torch.equal(out, fused)
    assert normwise(host(out), O.interpolate3(dst, src, f)) <= 1e-5


@pytest.mark.parametrize("B,Nd,Ns,C,relu,inplace", [(2, 4096, 1024, 128, True, True), (3, 100, 17, 5, True, False),
                                                    (2, 300, 50, 12, False, False), (1, 64, 16, 256, True, True)])
def test_interpolate3_add(gpu, B, Nd, Ns, C, relu, inplace):
    """phi(interpolation + add): the apply form's interpolation plus one
    addition, against the oracle's interpolation (1e-5); in place on add
    when asked, elementwise and strided (C = 5: element path)."""
    rr = g(16)
    dst = rr.uniform(-1, 1, (B, Nd, 3)).astype(np.float32)
    src = rr.uniform(-1, 1, (B, Ns, 3)).astype(np.float32)
    f = rr.standard_normal((B, Ns, C)).astype(np.float32)
    a = rr.standard_normal((B, Nd, C)).astype(np.float32)
    ref = O.interpolate3(dst, src, f).astype(np.float64) + a
    if relu:
        ref = np.maximum(ref, 0.0)
    nit, dist = ops.three_nn(dev(dst), dev(src))
    add = dev(a)
    out = ops.interpolate3_add(nit, dist, dev(f), add, relu=relu, out=add if inplace else None)
    assert (out.data_ptr() == add.data_ptr()) == inplace
    assert normwise(host(out), ref) <= 1e-5
    # the same as the apply form's output plus the addition, in fp32
    plain = host(ops.interpolate3_apply(nit, dist, dev(f))) + a
    assert np.array_equal(host(out), np.maximum(plain, 0.0) if relu else plain)


@pytest.mark.parametrize("B,Nd,Ns,widths", [(16, 4096, 1024, [128, 128, 128]), (3, 1000, 77, [20, 33, 9]),
                                             (2, 20000, 500, [64, 128, 13]),
                                             # weights beyond the LDS: staged in phases, one tile per wave
                                             (16, 4096, 1024, [128, 128, 128, 128, 13]),
                                             (2, 20001, 300, [128, 128, 128, 128, 128, 36])])
def test_interpolate3_mlp(gpu, B, Nd, Ns, widths):
    """The interpolate-add in the register MLP's loader: the two-call form's
    rows (mesorasi_interpolate3_add) bit for bit, so the same MLP gives the
    same output when that form also runs the register MLP (more than 32768
    rows); the oracle's interpolation + add + ReLU + MLP within 1e-4."""
    rr = g(17)
    C = widths[0]
    dst = rr.uniform(-1, 1, (B, Nd, 3)).astype(np.float32)
    src = rr.uniform(-1, 1, (B, Ns, 3)).astype(np.float32)
    f = rr.standard_normal((B, Ns, C)).astype(np.float32)
    a = rr.standard_normal((B, Nd, C)).astype(np.float32)
    Ws, bs = _weights(rr, widths)
    relu_mask = (1 << (len(widths) - 2)) - 1       # last layer linear
    p = ops.MLPParams(Ws, bs)
    assert ops.interpolate3_mlp_supported(p, B * Nd)
    nit, dist = ops.three_nn(dev(dst), dev(src))
    y = ops.interpolate3_mlp(nit, dist, dev(f), dev(a), p, relu_mask=relu_mask)
    h = ops.interpolate3_add(nit, dist, dev(f), dev(a))
    y2 = ops.pointwise_mlp(h, p, relu_mask=relu_mask)
    if B * Nd > 32768:
        assert torch.equal(y, y2)
    hr = np.maximum(O.interpolate3(dst, src, f).astype(np.float64) + a, 0.0).astype(np.float32)
    ref = O.mlp(hr.reshape(-1, C), Ws, bs, relu_mask=relu_mask).reshape(B, Nd, -1)
    assert normwise(host(y), ref) <= 1e-4


def test_three_nn_hand_example(gpu):
    """The hand-worked interpolation (weights 1/d2 over the 3 nearest)
    through the split GPU form."""
    d = json.load(open(os.path.join(GOLD, "interpolate3_weights.json")))
    dst = np.array([d["dst"]], np.float32)
    src = np.array([d["src"]], np.float32)
    f = np.array([d["features"]], np.float32)
    nit, dist = ops.three_nn(dev(dst), dev(src))
    assert host(nit).tolist() == [[[0, 1, 2]]]
    out = host(ops.interpolate3_apply(nit, dist, dev(f)))[0, 0].astype(np.float64)
    assert np.max(np.abs(out - np.array(d["expected_num"]) / d["expected_den"])) <= 1e-6


def test_interpolate3_overflowing_distances(gpu):
    """Sources beyond 1e20 (squared distances +inf, weight 0) beside two
    near sources: the 3-NN list still takes the lowest-index infinite
    source as its third entry, and the result is the two near sources'
    weighted mean."""
    rr = g(14)
    Ns, Nd = 1500, 70
    far = 1e20 * rr.uniform(1, 2, (1, Ns, 3)) * rr.choice([-1.0, 1.0], (1, Ns, 3))
    src = far.astype(np.float32)
    src[0, 5] = (0.1, 0.2, 0.3)
    src[0, 1100] = (-0.4, 0.0, 0.5)           # in the second staged chunk
    dst = rr.uniform(-1, 1, (1, Nd, 3)).astype(np.float32)
    f = rr.standard_normal((1, Ns, 8)).astype(np.float32)
    nn, dd = O.knn(src, dst, 3)
    assert (nn[..., :2] != 0).all() and np.isinf(dd[..., 2]).all()
    ref = O.interpolate3(dst, src, f)
    out = ops.interpolate3(dev(dst), dev(src), dev(f))
    assert normwise(host(out), ref) <= 1e-5


def test_cast_bf16_matches_oracle_rounding(gpu):
    rr = g(13)
    x = (rr.standard_normal(5000) * 10.0 ** rr.integers(-5, 5, 5000)).astype(np.float32)
    y = ops.cast_bf16(dev(x))
    assert np.array_equal(host(y.float()), O.bf16_round(x))


def test_edgeconv_fold(gpu):
    rr = g(14)
    W = rr.standard_normal((16, 10)).astype(np.float32)
    b = rr.standard_normal(16).astype(np.float32)
    from oracle.nets import edgeconv_fold as ofold
    rW, rb = ofold(W, b)
    Wo, bo = ops.edgeconv_fold(dev(W), dev(b))
    assert np.array_equal(host(Wo), rW) and np.array_equal(host(bo), rb)


def test_empty_batches_are_noops(gpu):
    x = torch.zeros((0, 10, 3), device="cuda")
    idx, cxyz = ops.fps(x, 5)
    assert idx.shape == (0, 5)
    nit, _ = ops.ball_query(torch.zeros((2, 10, 3), device="cuda"), torch.zeros((2, 0, 3), device="cuda"), 0.1, 4)
    assert nit.shape == (2, 0, 4)


# ----------------------------------------------------------------------------
# aggregation fused into the next module's MLP loader
# ----------------------------------------------------------------------------

AGG_MLP_CASES = {
    "seg_sa1_to_sa2": (16, 4096, 1024, 32, 64, [67, 64, 64, 128]),
    "ragged": (3, 500, 77, 5, 32, [35, 48, 40]),
    "c128_k64": (2, 1024, 300, 64, 128, [131, 128, 128, 128]),
}


@pytest.mark.parametrize("case", list(AGG_MLP_CASES), ids=list(AGG_MLP_CASES))
def test_aggregate_mlp_equals_aggregate_then_mlp(gpu, case):
    """The loader-side aggregation stores exactly mesorasi_aggregate_max's
    rows and feeds the same MLP kernel, so both outputs are identical to the
    two-kernel composition; the MLP output meets the oracle's tolerance."""
    B, N, M, K, C, dims = AGG_MLP_CASES[case]
    rr = g(16)
    pft = np.maximum(rr.standard_normal((B, N, C)), 0).astype(np.float32)
    nit = rr.integers(0, N, (B, M, K)).astype(np.int32)
    cidx = rr.integers(0, N, (B, M)).astype(np.int32)
    cxyz = rr.uniform(-1, 1, (B, M, 3)).astype(np.float32)
    Ws, bs = _weights(rr, dims)
    p = ops.MLPParams(Ws, bs)
    agg = torch.empty((B, M, C), device="cuda")
    y = ops.aggregate_mlp(dev(cxyz), dev(pft), dev(nit), dev(cidx), p, agg_out=agg)
    ref_agg = ops.aggregate_max(dev(pft), dev(nit), cidx=dev(cidx))
    ref_y = ops.pointwise_mlp(dev(cxyz), p, x1=ref_agg)
    assert torch.equal(agg, ref_agg)
    assert torch.equal(y.view(B * M, -1), ref_y.view(B * M, -1))
    o_agg = O.aggregate_max(pft, nit, cidx=cidx, sign=-1)
    assert np.array_equal(host(agg), o_agg)
    o_y = O.mlp(np.concatenate([cxyz, o_agg], -1), Ws, bs)
    assert normwise(host(y), o_y) <= 1e-4

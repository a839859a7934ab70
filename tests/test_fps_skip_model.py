"""CPU model of the skipping FPS form (clouds of 8193 to 16384 points),
checked against the oracle.

The form orders the cloud by the Morton code of its cell in a 16^3 grid over
the cloud's box, gives each thread P consecutive points of that order and
skips a wave's update when, for every thread of the wave, the distance bound
to the thread's box is at least the thread's largest running minimum.  The
bound applies the distance's own operations, in the same order, to the
per-axis gaps max(lo - c, c - hi, 0); since every operation is monotone in
its operands and each gap is at most the rounded |p - c|, the bound never
exceeds the distance an update would compute, so a skipped update changes
nothing.  These tests replay that argument in fp32 on the host:

  * the bound never exceeds the distance of any point of the box (random and
    adversarial boxes: points on the faces, the centroid inside, mixed
    signs, large and tiny magnitudes);
  * a full FPS with the skip rule (threads of P points, waves of 64 threads)
    selects exactly the oracle's points, and skips most updates on a
    clustered cloud.
"""
import numpy as np
import pytest

import oracle as O

f32 = np.float32


def _fma(a, b, c):
    # fp32 fma emulated through float64 (a * b exact there); the double
    # rounding is monotone too, which is all the argument uses
    return (a.astype(np.float64) * b.astype(np.float64) + c.astype(np.float64)).astype(f32)


def _dist(p, c):
    # t = p - c per axis, d = t_x^2, d = fma(t_y, t_y, d), d = fma(t_z, t_z, d)
    t = (p - c).astype(f32)
    d = (t[..., 0] * t[..., 0]).astype(f32)
    d = _fma(t[..., 1], t[..., 1], d)
    return _fma(t[..., 2], t[..., 2], d)


def _bound(lo, hi, c):
    g = np.maximum(np.maximum((lo - c).astype(f32), (c - hi).astype(f32)), f32(0))
    d = (g[..., 0] * g[..., 0]).astype(f32)
    d = _fma(g[..., 1], g[..., 1], d)
    return _fma(g[..., 2], g[..., 2], d)


@pytest.mark.parametrize("scale", [1.0, 1e-20, 1e18, 50.0])
def test_box_bound_never_exceeds_point_distance(scale):
    r = np.random.default_rng(5)
    for _ in range(200):
        pts = (r.standard_normal((16, 3)) * scale).astype(f32)
        if r.random() < 0.3:                       # points on the box faces
            pts[:3] = pts[:3].min(0)
            pts[3:6] = pts[3:6].max(0)
        lo, hi = pts.min(0), pts.max(0)
        cs = np.concatenate([(r.standard_normal((64, 3)) * scale * r.choice([0.1, 1, 10])).astype(f32),
                             pts[:4], ((lo + hi) / f32(2))[None], lo[None], hi[None]])
        with np.errstate(over="ignore"):   # squares of 1e19 overflow to inf on both sides
            for c in cs:
                assert np.all(_bound(lo, hi, c) <= _dist(pts, c))


def _morton_order(p):
    lo, hi = p.min(0), p.max(0)
    ext = hi - lo
    inv = np.where(ext > 0, f32(16) / np.where(ext > 0, ext, 1), 0).astype(f32)
    cell = np.clip(((p - lo) * inv).astype(f32), 0, 15).astype(np.int64)
    code = np.zeros(len(p), np.int64)
    for bit in range(4):
        for axis in range(3):
            code |= ((cell[:, axis] >> bit) & 1) << (3 * bit + axis)
    return np.argsort(code, kind="stable")


def _fps_skip(p, M, P=16):
    """FPS with the skip rule, ties to the lowest original index."""
    N = len(p)
    order = _morton_order(p)
    T = -(-N // P)
    W = -(-T // 64)
    slots = np.full(W * 64 * P, -1, np.int64)
    slots[:N] = order
    slots = slots.reshape(W, 64, P)
    slots.sort(axis=2)                                 # a thread's points ascend in index
    slots = np.where(slots < 0, -1, slots)
    real = slots >= 0
    pts = np.where(real[..., None], p[np.maximum(slots, 0)], f32(0))
    big = np.float32(np.inf)
    lo = np.where(real[..., None], pts, big).min(axis=2)
    hi = np.where(real[..., None], pts, -big).max(axis=2)
    dm = np.where(real, big, f32(-1))
    tmax = dm.max(axis=2)
    out = [0]
    c = p[0]
    skipped = 0
    for _ in range(1, M):
        lb = _bound(lo, hi, c)
        for w in range(W):
            if not np.any(lb[w] < tmax[w]):
                skipped += 1
                continue
            d = _dist(pts[w], c)
            dm[w] = np.where(real[w], np.minimum(dm[w], d), dm[w])
            tmax[w] = dm[w].max(axis=1)
        best = dm.max()
        j = int(slots[dm == best].min())               # lowest original index on ties
        out.append(j)
        c = p[j]
    return np.array(out, np.int32), skipped / (W * (M - 1))


@pytest.mark.parametrize("kind", ["clusters", "grid", "dups"])
def test_skip_rule_matches_oracle(kind):
    r = np.random.default_rng(9)
    N, M = 2000, 200
    if kind == "clusters":
        centres = r.standard_normal((8, 3)).astype(f32) * 4
        p = (centres[r.integers(0, 8, N)] + r.standard_normal((N, 3)).astype(f32) * 0.3).astype(f32)
    elif kind == "grid":
        p = r.integers(0, 4, size=(N, 3)).astype(f32)
    else:
        base = r.standard_normal((N // 5, 3)).astype(f32)
        p = base[r.integers(0, N // 5, N)]
    idx, frac = _fps_skip(p, M, P=4)
    ref, _ = O.fps(p[None], M)
    assert np.array_equal(idx, ref[0])
    if kind == "clusters":
        assert frac > 0.3                              # the rule does skip on spatially coherent clouds

"""Seeded synthetic inputs: point clouds, extra features and MLP weights.

This module only draws random numbers and shapes geometry; it holds none of
the delayed-aggregation arithmetic (no sampling, search, MLP or aggregation).
Both the HIP path and the CPU oracle are fed from here, so a parity test
hands the very same arrays to each side.

Every generator takes a numpy Generator built by :func:`rng`, seeded from
``SeedSequence([200806967, config_id, stream])`` with streams
0 = points, 1 = extra features, 2 = weights, 3 = biases, 4+ = test-specific.

Workload stand-ins (the paper's datasets are not used; nothing here
reproduces any item of them):
  * ``uniform_cube``   - points uniform in [-1, 1]^3 (single-module case).
  * ``mesh_surfaces``  - ModelNet40-like objects: a union of 1-4 spheres,
    boxes and cylinders sampled area-uniformly, centred and scaled to unit
    max-norm (the 1024-point objects of the paper's classification nets).
  * ``indoor_room``    - scene-segmentation-like rooms: floor, 2-4 walls and
    3-8 clusters of 2-6 boxes, with 3 extra per-point features in [0, 1].
  * ``lidar_scene``    - KITTI-like 64-ring LiDAR sweeps over a ground plane
    and 30 boxes, strongly non-uniform density (the paper's 130K-point
    frames, sub-sampled to 16384 points).
"""
from __future__ import annotations

import numpy as np

SEED_ROOT = 200806967


def rng(config_id: int, stream: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([SEED_ROOT, int(config_id), int(stream)]))


# ----------------------------------------------------------------------------
# geometry helpers (float64 internally, float32 on output)
# ----------------------------------------------------------------------------

def _random_rotation(g: np.random.Generator) -> np.ndarray:
    q, r = np.linalg.qr(g.standard_normal((3, 3)))
    q = q * np.sign(np.diag(r))
    if np.linalg.det(q) < 0:
        q[:, 0] = -q[:, 0]
    return q


def _sample_sphere(g, n, radius):
    v = g.standard_normal((n, 3))
    v /= np.linalg.norm(v, axis=1, keepdims=True)
    return v * radius


def _box_faces(sides):
    """Six faces of an axis-aligned box centred at 0: (areas, sampler)."""
    a, b, c = sides
    return np.array([b * c, b * c, a * c, a * c, a * b, a * b])


def _sample_box(g, n, sides):
    sides = np.asarray(sides, dtype=np.float64)
    areas = _box_faces(sides)
    face = g.choice(6, size=n, p=areas / areas.sum())
    u = g.uniform(-0.5, 0.5, size=(n, 3)) * sides
    axis = face // 2
    sign = np.where(face % 2 == 0, -0.5, 0.5)
    u[np.arange(n), axis] = sign * sides[axis]
    return u


def _sample_cylinder(g, n, radius, height):
    side = 2 * np.pi * radius * height
    cap = np.pi * radius * radius
    part = g.choice(3, size=n, p=np.array([side, cap, cap]) / (side + 2 * cap))
    theta = g.uniform(0, 2 * np.pi, size=n)
    out = np.empty((n, 3))
    # lateral surface
    out[:, 0] = radius * np.cos(theta)
    out[:, 1] = radius * np.sin(theta)
    out[:, 2] = g.uniform(-height / 2, height / 2, size=n)
    # caps: area-uniform disc sampling
    caps = part > 0
    rr = radius * np.sqrt(g.uniform(0, 1, size=n))
    out[caps, 0] = rr[caps] * np.cos(theta[caps])
    out[caps, 1] = rr[caps] * np.sin(theta[caps])
    out[caps, 2] = np.where(part[caps] == 1, -height / 2, height / 2)
    return out


def _primitive_area(kind, size):
    if kind == 0:
        return 4 * np.pi * size[0] ** 2
    if kind == 1:
        return float(_box_faces(size).sum())
    r, h = size[0], size[1]
    return 2 * np.pi * r * h + 2 * np.pi * r * r


# ----------------------------------------------------------------------------
# point-cloud generators
# ----------------------------------------------------------------------------

def uniform_cube(g: np.random.Generator, B: int, N: int) -> np.ndarray:
    return g.uniform(-1.0, 1.0, size=(B, N, 3)).astype(np.float32)


def mesh_surfaces(g: np.random.Generator, B: int, N: int) -> np.ndarray:
    """Union of 1-4 primitives (sphere/box/cylinder, size in [0.2, 1]),
    randomly rotated and offset, N points sampled area-uniformly, centred on
    the mean and scaled to max-norm 1."""
    out = np.empty((B, N, 3), dtype=np.float32)
    for b in range(B):
        n_prim = int(g.integers(1, 5))
        kinds = g.integers(0, 3, size=n_prim)
        sizes = [g.uniform(0.2, 1.0, size=3) for _ in range(n_prim)]
        # sphere: radius = s/2; box: sides = s; cylinder: radius s0/2, height s1
        geo = []
        for k, s in zip(kinds, sizes):
            if k == 0:
                geo.append((0, np.array([s[0] / 2])))
            elif k == 1:
                geo.append((1, s))
            else:
                geo.append((2, np.array([s[0] / 2, s[1]])))
        areas = np.array([_primitive_area(k, s) for k, s in geo])
        counts = g.multinomial(N, areas / areas.sum())
        pts = []
        for (k, s), c in zip(geo, counts):
            if c == 0:
                continue
            if k == 0:
                p = _sample_sphere(g, c, s[0])
            elif k == 1:
                p = _sample_box(g, c, s)
            else:
                p = _sample_cylinder(g, c, s[0], s[1])
            p = p @ _random_rotation(g).T + g.uniform(-0.5, 0.5, size=3)
            pts.append(p)
        p = np.concatenate(pts, axis=0)
        p = p[g.permutation(N)]
        p -= p.mean(axis=0)
        p /= np.max(np.linalg.norm(p, axis=1))
        out[b] = p.astype(np.float32)
    return out


def indoor_room(g: np.random.Generator, B: int, N: int, n_feat: int = 3):
    """Room layouts: floor (z=0), 2-4 walls, 3-8 clusters of 2-6 boxes, all
    sampled area-uniformly; x, y centred and scaled into [-1, 1], z >= 0
    scaled by the same factor.  Returns (xyz [B,N,3], feat [B,N,n_feat])
    with features uniform in [0, 1]."""
    xyz = np.empty((B, N, 3), dtype=np.float32)
    for b in range(B):
        L = g.uniform(4.0, 8.0, size=2)
        H = g.uniform(2.5, 3.5)
        # surfaces: (area, sampler)
        surfaces = []
        surfaces.append((L[0] * L[1], lambda n, L=L: np.stack(
            [g.uniform(-L[0] / 2, L[0] / 2, n), g.uniform(-L[1] / 2, L[1] / 2, n), np.zeros(n)], 1)))
        walls = g.permutation(4)[: int(g.integers(2, 5))]
        for w in walls:
            if w < 2:  # wall at x = +-L0/2 spanning y
                x0 = (-1 if w == 0 else 1) * L[0] / 2
                surfaces.append((L[1] * H, lambda n, x0=x0, L=L: np.stack(
                    [np.full(n, x0), g.uniform(-L[1] / 2, L[1] / 2, n), g.uniform(0, H, n)], 1)))
            else:
                y0 = (-1 if w == 2 else 1) * L[1] / 2
                surfaces.append((L[0] * H, lambda n, y0=y0, L=L: np.stack(
                    [g.uniform(-L[0] / 2, L[0] / 2, n), np.full(n, y0), g.uniform(0, H, n)], 1)))
        for _ in range(int(g.integers(3, 9))):
            cc = g.uniform(-0.4, 0.4, size=2) * L
            for _ in range(int(g.integers(2, 7))):
                sides = g.uniform(0.2, 1.5, size=3)
                centre = np.array([cc[0] + g.uniform(-0.7, 0.7), cc[1] + g.uniform(-0.7, 0.7), sides[2] / 2])
                yaw = g.uniform(0, 2 * np.pi)
                rot = np.array([[np.cos(yaw), -np.sin(yaw), 0], [np.sin(yaw), np.cos(yaw), 0], [0, 0, 1]])
                surfaces.append((float(_box_faces(sides).sum()),
                                 lambda n, s=sides, c=centre, R=rot: _sample_box(g, n, s) @ R.T + c))
        areas = np.array([a for a, _ in surfaces])
        counts = g.multinomial(N, areas / areas.sum())
        pts = np.concatenate([f(c) for (a, f), c in zip(surfaces, counts) if c > 0], axis=0)
        pts = pts[g.permutation(N)]
        pts[:, :2] -= (pts[:, :2].max(0) + pts[:, :2].min(0)) / 2
        pts[:, 2] -= pts[:, 2].min()
        pts /= np.abs(pts[:, :2]).max()
        xyz[b] = pts.astype(np.float32)
    feat = g.uniform(0.0, 1.0, size=(B, N, n_feat)).astype(np.float32)
    return xyz, feat


def _ray_box_hits(origin, dirs, centre, half, yaw):
    """Slab intersection of rays with one yaw-rotated box: entry distance or inf."""
    c, s = np.cos(-yaw), np.sin(-yaw)
    rot = np.array([[c, -s, 0], [s, c, 0], [0, 0, 1]])
    o = rot @ (origin - centre)
    d = dirs @ rot.T
    with np.errstate(divide="ignore", invalid="ignore"):
        inv = 1.0 / d
        t1 = (-half - o) * inv
        t2 = (half - o) * inv
    tmin = np.nanmax(np.minimum(t1, t2), axis=1)
    tmax = np.nanmin(np.maximum(t1, t2), axis=1)
    hit = (tmax >= np.maximum(tmin, 0.0))
    t = np.where(tmin > 0, tmin, tmax)
    return np.where(hit & (t > 0), t, np.inf)


def lidar_scene(g: np.random.Generator, B: int, N: int, rings: int = 64, azimuths: int = 1024,
                max_range: float = 50.0, n_boxes: int = 30):
    """A 64-ring spinning LiDAR at 1.7 m over ground z=0 with 30 yaw-rotated
    boxes (sides 0.5-4.5 m, centres 5-40 m away); first-return ray casting,
    range noise N(0, 0.02 m), returns beyond 50 m dropped, exactly N returns
    drawn without replacement, coordinates divided by 50 m."""
    out = np.empty((B, N, 3), dtype=np.float32)
    elev = np.deg2rad(np.linspace(-24.8, 2.0, rings))
    sensor = np.array([0.0, 0.0, 1.7])
    for b in range(B):
        az = (np.arange(azimuths)[None, :] * (2 * np.pi / azimuths)
              + g.uniform(0, 2 * np.pi / azimuths, size=(rings, 1)))
        el = np.broadcast_to(elev[:, None], az.shape)
        dirs = np.stack([np.cos(el) * np.cos(az), np.cos(el) * np.sin(az), np.sin(el)], -1).reshape(-1, 3)
        with np.errstate(divide="ignore"):
            t_ground = np.where(dirs[:, 2] < 0, -sensor[2] / dirs[:, 2], np.inf)
        t = t_ground
        for _ in range(n_boxes):
            rad = g.uniform(5.0, 40.0)
            ang = g.uniform(0, 2 * np.pi)
            sides = g.uniform(0.5, 4.5, size=3)
            centre = np.array([rad * np.cos(ang), rad * np.sin(ang), sides[2] / 2])
            t = np.minimum(t, _ray_box_hits(sensor, dirs, centre, sides / 2, g.uniform(0, 2 * np.pi)))
        t = t + g.normal(0.0, 0.02, size=t.shape)
        ok = np.isfinite(t) & (t > 0) & (t <= max_range)
        pts = sensor + dirs[ok] * t[ok, None]
        if pts.shape[0] < N:
            raise ValueError(f"only {pts.shape[0]} returns, need {N}")
        pick = g.choice(pts.shape[0], size=N, replace=False)
        out[b] = (pts[pick] / max_range).astype(np.float32)
    return out


# ----------------------------------------------------------------------------
# weights
# ----------------------------------------------------------------------------

def he_layers(g_w: np.random.Generator, g_b: np.random.Generator, dims):
    """He-normal weights N(0, 2/fan_in) as [C_out, C_in] float32 (the torch
    Linear / 1x1-conv layout) and biases uniform in [-0.1, 0.1]."""
    Ws, bs = [], []
    for cin, cout in zip(dims[:-1], dims[1:]):
        Ws.append((g_w.standard_normal((cout, cin)) * np.sqrt(2.0 / cin)).astype(np.float32))
        bs.append(g_b.uniform(-0.1, 0.1, size=cout).astype(np.float32))
    return Ws, bs


# ----------------------------------------------------------------------------
# the five synthetic workloads: shapes and hyper-parameters only
# ----------------------------------------------------------------------------

def _sa(M, radius, K, mlp):
    return dict(M=M, radius=radius, K=K, mlp=list(mlp))


WORKLOADS = {
    # one set-abstraction module, the paper's walk-through shape
    # (1024 -> 512 centroids, K = 32, 3 -> 128; Sec. 4.1)
    "sa_module": dict(id=0, kind="pointnet2_cls", B=1, N=1024, gen="uniform_cube", n_feat=0,
                      sa=[_sa(512, 0.2, 32, [64, 64, 128])], group_all=None, fc=None, dtype="f32"),
    # PointNet++ SSG classifier (ModelNet40-like objects)
    "pointnet2_cls": dict(id=1, kind="pointnet2_cls", B=32, N=1024, gen="mesh_surfaces", n_feat=0,
                          sa=[_sa(512, 0.2, 32, [64, 64, 128]), _sa(128, 0.4, 64, [128, 128, 256])],
                          group_all=[256, 512, 1024], fc=[512, 256, 40], dtype="f32"),
    # DGCNN EdgeConv stack
    "dgcnn": dict(id=2, kind="dgcnn", B=16, N=1024, gen="mesh_surfaces", n_feat=0, k=20,
                  edge=[64, 64, 128, 256], conv=1024, dtype="f32"),
    # PointNet++ segmentation of indoor rooms, xyz + 3 extra features
    "pointnet2_seg": dict(id=3, kind="pointnet2_seg", B=16, N=4096, gen="indoor_room", n_feat=3,
                          sa=[_sa(1024, 0.1, 32, [32, 32, 64]), _sa(256, 0.2, 32, [64, 64, 128]),
                              _sa(64, 0.4, 32, [128, 128, 256]), _sa(16, 0.8, 32, [256, 256, 512])],
                          fp=[[256, 256], [256, 256], [256, 128], [128, 128, 128]], head=[128, 13],
                          n_classes=13, dtype="f32"),
    # KITTI-like LiDAR scene, bf16 MLPs
    "lidar": dict(id=4, kind="pointnet2_cls", B=4, N=16384, gen="lidar_scene", n_feat=0,
                  sa=[_sa(4096, 0.1, 64, [32, 32, 64]), _sa(1024, 0.2, 64, [64, 64, 128]),
                      _sa(256, 0.4, 64, [128, 128, 256])], group_all=None, fc=None, dtype="bf16"),
}


def workload(name: str, **override) -> dict:
    """A copy of a workload spec, optionally with B/N/dtype overridden
    (smaller batches for tests; the bf16 variant of the segmentation net)."""
    import copy
    spec = copy.deepcopy(WORKLOADS[name])
    spec.update(override)
    spec["name"] = name
    return spec


def make_points(spec: dict):
    """(xyz [B,N,3] float32, feat [B,N,n_feat] float32 or None)."""
    g = rng(spec["id"], 0)
    B, N = spec["B"], spec["N"]
    if spec["gen"] == "uniform_cube":
        return uniform_cube(g, B, N), None
    if spec["gen"] == "mesh_surfaces":
        return mesh_surfaces(g, B, N), None
    if spec["gen"] == "indoor_room":
        xyz, _ = indoor_room(g, B, N, n_feat=0)
        feat = rng(spec["id"], 1).uniform(0.0, 1.0, size=(B, N, spec["n_feat"])).astype(np.float32)
        return xyz, feat
    if spec["gen"] == "lidar_scene":
        return lidar_scene(g, B, N), None
    raise ValueError(spec["gen"])


def make_weights(spec: dict) -> dict:
    """All layer weights of a workload, drawn in network order from the
    weight (2) and bias (3) streams.  Keys:
      sa:   list of (Ws, bs) per set-abstraction module
      group_all, fc, head: (Ws, bs)
      fp:   list of (Ws, bs) per feature-propagation module
      edge: list of (W [C_out, 2 C_in], b) per EdgeConv layer; conv: (W, b)
    """
    gw, gb = rng(spec["id"], 2), rng(spec["id"], 3)
    out = {}
    kind = spec["kind"]
    if kind in ("pointnet2_cls", "pointnet2_seg"):
        cin = 3 + spec["n_feat"]
        out["sa"] = []
        for m in spec["sa"]:
            out["sa"].append(he_layers(gw, gb, [cin] + m["mlp"]))
            cin = 3 + m["mlp"][-1]
        if spec.get("group_all"):
            out["group_all"] = he_layers(gw, gb, [cin] + spec["group_all"])
            cin = spec["group_all"][-1]
        if spec.get("fc"):
            out["fc"] = he_layers(gw, gb, [cin] + spec["fc"])
        if kind == "pointnet2_seg":
            widths = [3 + spec["n_feat"] - 3] + [m["mlp"][-1] for m in spec["sa"]]  # skip widths per level
            out["fp"] = []
            coarse = widths[-1]
            for i, dims in enumerate(spec["fp"]):
                skip = widths[len(widths) - 2 - i]
                out["fp"].append(he_layers(gw, gb, [coarse + skip] + dims))
                coarse = dims[-1]
            out["head"] = he_layers(gw, gb, [coarse] + spec["head"])
    elif kind == "dgcnn":
        cin = 3
        out["edge"] = []
        for cout in spec["edge"]:
            Ws, bs = he_layers(gw, gb, [2 * cin, cout])
            out["edge"].append((Ws[0], bs[0]))
            cin = cout
        Ws, bs = he_layers(gw, gb, [sum(spec["edge"]), spec["conv"]])
        out["conv"] = (Ws[0], bs[0])
    return out

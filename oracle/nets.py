"""Oracle compositions of the paper's modules and networks (test
infrastructure only; see the package docstring).

Each function takes plain numpy arrays plus the layer weights and returns
numpy arrays; every arithmetic step is one of the C primitives in
``oracle.c`` (numpy here only concatenates, slices and reshapes, except the
one-off EdgeConv weight fold ``fl32(W1 - W2)``, which is a float32 numpy
subtraction, i.e. one IEEE binary32 subtraction per element).

Delayed modules follow Sec. 4.1 (Eq. (2)-(3), walk-through): F runs once on
the N input points into the point feature table (PFT), N produces the
neighbor index table (NIT), and A gathers PFT rows by the NIT, reduces them
with max and then combines the centroid's own PFT row.  Conventional
modules follow Sec. 3.1 (Eq. (1)): N, then A builds the neighbor feature
matrix, then F on every (centroid, neighbor) row, then the max reduction.
"""
from __future__ import annotations

import numpy as np

from . import (fps, ball_query, knn, mlp, aggregate_max, group_pointnet, group_edge, rowgroup_max,
               interpolate3, ltd_group)


def _cat(xyz, feat):
    return xyz if feat is None else np.concatenate([xyz, feat], axis=-1)


def sa_delayed(xyz, feat, M, radius, K, Ws, bs, bf16=False):
    """Set-abstraction module with delayed aggregation."""
    idx, cxyz = fps(xyz, M)
    nit, cnt, _ = ball_query(xyz, cxyz, radius, K)
    pft = mlp(_cat(xyz, feat), Ws, bs, bf16=bf16)           # F on all N input points
    out = aggregate_max(pft, nit, cidx=idx, sign=-1)          # max_k PFT[nit] - PFT[centroid]
    return dict(idx=idx, cxyz=cxyz, nit=nit, cnt=cnt, pft=pft, out=out)


def sa_conventional(xyz, feat, M, radius, K, Ws, bs, bf16=False):
    """Set-abstraction module in the original order: N, A (NFM), F, max."""
    idx, cxyz = fps(xyz, M)
    nit, cnt, _ = ball_query(xyz, cxyz, radius, K)
    nfm = group_pointnet(xyz, feat, cxyz, nit)                # [B, M, K, 3 + cf]
    h = mlp(nfm, Ws, bs, bf16=bf16)                           # [B, M, K, C]
    B, C = xyz.shape[0], h.shape[-1]
    out = rowgroup_max(h.reshape(B, M * K, C), K)             # [B, M, C]
    return dict(idx=idx, cxyz=cxyz, nit=nit, cnt=cnt, out=out)


def sa_ltd(xyz, feat, M, radius, K, Ws, bs):
    """Set-abstraction module with limited delayed aggregation (Sec. 7.3):
    the first layer's matrix product runs once on the N input points (P1)
    and once on the centroids' coordinates with the xyz columns of W1 (Q);
    each (centroid, neighbor) row then starts from ReLU(P1[j] - Q[c] + b1)
    and the remaining layers run on the K neighbor rows before the max.
    Exact in real arithmetic: W1 [x_j - x_c | f_j] = W1 [x_j | f_j] -
    W1[:, :3] x_c."""
    idx, cxyz = fps(xyz, M)
    nit, cnt, _ = ball_query(xyz, cxyz, radius, K)
    W1 = np.asarray(Ws[0], np.float32)
    p1 = mlp(_cat(xyz, feat), [W1], [None], relu_mask=0)          # [B, N, C1]
    q = mlp(cxyz, [np.ascontiguousarray(W1[:, :3])], [None], relu_mask=0)   # [B, M, C1]
    h = ltd_group(p1, q, bs[0], nit)                              # [B, M, K, C1]
    if len(Ws) > 1:
        h = mlp(h, Ws[1:], bs[1:])
    B, C = xyz.shape[0], h.shape[-1]
    out = rowgroup_max(h.reshape(B, M * K, C), K)
    return dict(idx=idx, cxyz=cxyz, nit=nit, cnt=cnt, p1=p1, q=q, out=out)


def group_all(xyz, feat, Ws, bs, bf16=False):
    """Group-all module: MLP on every point then max over the cloud (no
    centroid term; identical in both orders)."""
    h = mlp(_cat(xyz, feat), Ws, bs, bf16=bf16)
    return rowgroup_max(h, h.shape[1])[:, 0, :]


def fc_head(x, Ws, bs, bf16=False):
    """Fully-connected layers, ReLU on all but the last."""
    n = len(Ws)
    return mlp(x, Ws, bs, relu_mask=(1 << (n - 1)) - 1, bf16=bf16)


def edgeconv_fold(W, b):
    """W [C_out, 2C] acting on [x_i, x_j - x_i] -> stacked weights
    [[W1 - W2], [W2]] of shape [2 C_out, C] and bias [b, 0]."""
    C = W.shape[1] // 2
    W1, W2 = W[:, :C], W[:, C:]
    Wd = (W1.astype(np.float32) - W2.astype(np.float32)).astype(np.float32)
    return np.concatenate([Wd, W2], 0).astype(np.float32), np.concatenate([b, np.zeros_like(b)]).astype(np.float32)


def edgeconv_delayed(X, k, W, b):
    """EdgeConv with delayed aggregation:
    out_i = ReLU(max_j W2 x_j + (W1 - W2) x_i + b)."""
    Cout = W.shape[0]
    nit, dist = knn(X, X, k)
    Ws, bs = edgeconv_fold(W, b)
    P = mlp(X, [Ws], [bs], relu_mask=0)                       # [B, N, 2 C_out]: A | Bm
    A, Bm = P[..., :Cout], P[..., Cout:]
    out = aggregate_max(Bm, nit, cfeat=A, sign=+1, relu=True)
    return dict(nit=nit, out=out)


def edgeconv_conventional(X, k, W, b):
    """EdgeConv in the original order: out_i = max_j ReLU(W [x_i, x_j - x_i] + b)."""
    B, N, _ = X.shape
    nit, dist = knn(X, X, k)
    nfm = group_edge(X, nit)                                  # [B, N, k, 2C]
    h = mlp(nfm, [W], [b])
    out = rowgroup_max(h.reshape(B, N * k, -1), k)
    return dict(nit=nit, out=out)


# ----------------------------------------------------------------------------
# networks
# ----------------------------------------------------------------------------

def _sa_order(delayed, bf16):
    """delayed: True (Sec. 4.1), False (conventional, Sec. 3.1) or "ltd"
    (limited delayed aggregation, Sec. 7.3; fp32 networks)."""
    if delayed == "ltd":
        if bf16:
            raise ValueError("the limited delayed order is composed for fp32 networks")
        return lambda p, f, M, r, K, Ws, bs, bf16=False: sa_ltd(p, f, M, r, K, Ws, bs)
    return sa_delayed if delayed else sa_conventional


def pointnet2_cls(spec, xyz, feat, weights, delayed=True):
    """Set-abstraction stack [+ group-all + FC head].  Returns a dict with
    per-module outputs and the final tensor under 'out'."""
    bf16 = spec["dtype"] == "bf16"
    sa = _sa_order(delayed, bf16)
    res = dict(modules=[])
    p, f = xyz, feat
    for m, (Ws, bs) in zip(spec["sa"], weights["sa"]):
        r = sa(p, f, m["M"], m["radius"], m["K"], Ws, bs, bf16=bf16)
        res["modules"].append(r)
        p, f = r["cxyz"], r["out"]
    res["out"] = f
    if spec.get("group_all"):
        g = group_all(p, f, *weights["group_all"], bf16=bf16)
        res["global"] = g
        res["out"] = g
        if spec.get("fc"):
            res["out"] = fc_head(g, *weights["fc"], bf16=bf16)
    return res


def dgcnn(spec, xyz, weights, delayed=True):
    """delayed=True or "ltd": the delayed EdgeConv.  Its module has one
    layer, so hoisting that layer's product (the limited order, Sec. 7.3)
    is the whole delayed order."""
    ec = edgeconv_delayed if delayed else edgeconv_conventional
    X = xyz
    res = dict(layers=[])
    outs = []
    for W, b in weights["edge"]:
        r = ec(X, spec["k"], W, b)
        res["layers"].append(r)
        outs.append(r["out"])
        X = r["out"]
    cat = np.concatenate(outs, axis=-1)
    Wc, bc = weights["conv"]
    h = mlp(cat, [Wc], [bc])
    res["out"] = rowgroup_max(h, h.shape[1])[:, 0, :]
    return res


def pointnet2_seg(spec, xyz, feat, weights, delayed=True):
    bf16 = spec["dtype"] == "bf16"
    sa = _sa_order(delayed, bf16)
    levels = [(xyz, feat)]
    res = dict(modules=[], fp=[])
    p, f = xyz, feat
    for m, (Ws, bs) in zip(spec["sa"], weights["sa"]):
        r = sa(p, f, m["M"], m["radius"], m["K"], Ws, bs, bf16=bf16)
        res["modules"].append(r)
        p, f = r["cxyz"], r["out"]
        levels.append((p, f))
    coarse_xyz, coarse_f = levels[-1]
    for i, (Ws, bs) in enumerate(weights["fp"]):
        fine_xyz, fine_f = levels[len(levels) - 2 - i]
        interp = interpolate3(fine_xyz, coarse_xyz, coarse_f)
        x = interp if fine_f is None else np.concatenate([interp, fine_f], axis=-1)
        coarse_f = mlp(x, Ws, bs, bf16=bf16)
        coarse_xyz = fine_xyz
        res["fp"].append(coarse_f)
    res["out"] = fc_head(coarse_f, *weights["head"], bf16=bf16)
    return res


def forward(spec, xyz, feat, weights, delayed=True):
    if spec["kind"] == "pointnet2_cls":
        return pointnet2_cls(spec, xyz, feat, weights, delayed)
    if spec["kind"] == "dgcnn":
        return dgcnn(spec, xyz, weights, delayed)
    if spec["kind"] == "pointnet2_seg":
        return pointnet2_seg(spec, xyz, feat, weights, delayed)
    raise ValueError(spec["kind"])

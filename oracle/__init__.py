"""CPU oracle for the delayed-aggregation hot path.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
CPU-baseline leg of the benchmark may import this package.  The product
path (``paper_2008_06967_amd``) never imports, loads or calls it, and it
imports nothing from the product path: both sides are only ever fed the
same arrays from the seeded generators.

The arithmetic lives in ``oracle.c`` (plain scalar C, single thread); this
module marshals numpy arrays into it.  ``nets`` composes the primitives into
the paper's modules and networks.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from .build import build as _build, LIB_PATH

_lib = None

_i64 = ctypes.c_int64
_i32 = ctypes.c_int32
_p = ctypes.c_void_p


def lib():
    global _lib
    if _lib is None:
        # MESORASI_ORACLE_LIBRARY: the same oracle.c built with sanitizers
        path = os.environ.get("MESORASI_ORACLE_LIBRARY") or LIB_PATH
        if path == LIB_PATH and not os.path.exists(LIB_PATH):
            _build()
        L = ctypes.CDLL(path)
        L.orc_dist2.restype = ctypes.c_float
        L.orc_dist2.argtypes = [_p, _p, ctypes.c_int]
        L.orc_bf16_round.restype = ctypes.c_float
        L.orc_bf16_round.argtypes = [ctypes.c_float]
        L.orc_fps.argtypes = [_p, _i64, _i64, _i64, _p, _p]
        L.orc_fps_bruteforce.argtypes = [_p, _i64, _i64, _i64, _p]
        L.orc_ball_query.argtypes = [_p, _p, _i64, _i64, _i64, ctypes.c_float, _i32, _p, _p, _p]
        L.orc_knn.argtypes = [_p, _i64, _p, _i64, _i64, _i64, _i64, _i32, _i32, _p, _p]
        L.orc_mlp.argtypes = [_p, _i64, _i32, _p, _p, _p, ctypes.c_uint32, _i32, _p]
        L.orc_aggregate_max.argtypes = [_p, _i64, _p, _i64, _i64, _i64, _i32, _i32, _p, _p, _i64, _i32, _i32,
                                        _p, _i64]
        L.orc_group_pointnet.argtypes = [_p, _p, _i32, _i64, _p, _p, _i64, _i64, _i64, _i32, _p]
        L.orc_group_offsets.argtypes = [_p, _p, _i32, _i64, _p, _p, _i64, _i64, _i64, _i32, _p]
        L.orc_group_edge.argtypes = [_p, _i64, _i32, _p, _i64, _i64, _i32, _p]
        L.orc_rowgroup_max.argtypes = [_p, _i64, _i32, _i32, _p, _i64]
        L.orc_interpolate3.argtypes = [_p, _p, _p, _i64, _i64, _i64, _i64, _i32, _p, _i64]
        L.orc_ltd_group.argtypes = [_p, _p, _p, _p, _i64, _i64, _i64, _i32, _i32, _p]
        for fn in ("orc_fps", "orc_fps_bruteforce", "orc_ball_query", "orc_knn", "orc_mlp", "orc_aggregate_max",
                   "orc_group_pointnet", "orc_group_offsets", "orc_group_edge", "orc_rowgroup_max", "orc_ltd_group",
                   "orc_interpolate3"):
            getattr(L, fn).restype = None
        _lib = L
    return _lib


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def _i32a(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def _ptr(a):
    return None if a is None else a.ctypes.data


# ----------------------------------------------------------------------------
# primitives
# ----------------------------------------------------------------------------

def dist2(a, b) -> np.float32:
    a, b = _f32(a), _f32(b)
    return np.float32(lib().orc_dist2(_ptr(a), _ptr(b), a.shape[-1]))


def bf16_round(x):
    """fp32 -> bf16 (round to nearest even) -> fp32, elementwise."""
    x = _f32(x)
    f = lib().orc_bf16_round
    return np.array([f(float(v)) for v in x.reshape(-1)], dtype=np.float32).reshape(x.shape)


def fps(xyz, M):
    """xyz [B,N,3] -> (idx int32 [B,M], cxyz float32 [B,M,3])."""
    xyz = _f32(xyz)
    B, N, _ = xyz.shape
    idx = np.empty((B, M), np.int32)
    cxyz = np.empty((B, M, 3), np.float32)
    lib().orc_fps(_ptr(xyz), B, N, M, _ptr(idx), _ptr(cxyz))
    return idx, cxyz


def fps_bruteforce(xyz, M):
    xyz = _f32(xyz)
    B, N, _ = xyz.shape
    idx = np.empty((B, M), np.int32)
    lib().orc_fps_bruteforce(_ptr(xyz), B, N, M, _ptr(idx))
    return idx


def ball_query(xyz, qxyz, radius, K):
    """-> (nit int32 [B,M,K], cnt int32 [B,M], scanned int64 [B,M])."""
    xyz, qxyz = _f32(xyz), _f32(qxyz)
    B, N, _ = xyz.shape
    M = qxyz.shape[1]
    nit = np.empty((B, M, K), np.int32)
    cnt = np.empty((B, M), np.int32)
    scanned = np.empty((B, M), np.int64)
    lib().orc_ball_query(_ptr(xyz), _ptr(qxyz), B, N, M, np.float32(radius), K, _ptr(nit), _ptr(cnt),
                         _ptr(scanned))
    return nit, cnt, scanned


def knn(ref, query, K):
    """ref [B,N,C], query [B,M,C] -> (nit int32 [B,M,K], dist float32 [B,M,K])."""
    ref, query = _f32(ref), _f32(query)
    B, N, C = ref.shape
    M = query.shape[1]
    nit = np.empty((B, M, K), np.int32)
    dist = np.empty((B, M, K), np.float32)
    lib().orc_knn(_ptr(ref), C, _ptr(query), C, B, N, M, C, K, _ptr(nit), _ptr(dist))
    return nit, dist


def mlp(x, Ws, bs, relu_mask=None, bf16=False):
    """x [..., C0]; Ws[l] [C_{l+1}, C_l]; bs[l] [C_{l+1}] or None."""
    x = _f32(x)
    lead = x.shape[:-1]
    rows = int(np.prod(lead)) if lead else 1
    n = len(Ws)
    dims = [x.shape[-1]] + [int(W.shape[0]) for W in Ws]
    for l, W in enumerate(Ws):
        assert W.shape == (dims[l + 1], dims[l]), (W.shape, dims)
    if relu_mask is None:
        relu_mask = (1 << n) - 1
    Wc = [_f32(W) for W in Ws]
    bc = [None if b is None else _f32(b) for b in bs]
    dims_a = np.array(dims, np.int32)
    Wp = (ctypes.c_void_p * n)(*[_ptr(W) for W in Wc])
    bp = (ctypes.c_void_p * n)(*[_ptr(b) for b in bc])
    y = np.empty((rows, dims[-1]), np.float32)
    lib().orc_mlp(_ptr(x), rows, n, _ptr(dims_a), ctypes.cast(Wp, ctypes.c_void_p),
                  ctypes.cast(bp, ctypes.c_void_p), relu_mask, 1 if bf16 else 0, _ptr(y))
    return y.reshape(lead + (dims[-1],))


def ltd_group(p1, q, b1, nit):
    """p1 [B,N,C]; q [B,M,C]; b1 [C] or None; nit [B,M,K] -> h1 [B,M,K,C] =
    ReLU(p1[nit] - q + b1) (the first layer of a limited-delayed module)."""
    p1, q, nit = _f32(p1), _f32(q), _i32a(nit)
    B, N, C = p1.shape
    M, K = nit.shape[1], nit.shape[2]
    assert q.shape == (B, M, C)
    bb = None if b1 is None else _f32(b1)
    h1 = np.empty((B, M, K, C), np.float32)
    lib().orc_ltd_group(_ptr(p1), _ptr(q), _ptr(bb), _ptr(nit), B, N, M, K, C, _ptr(h1))
    return h1


def aggregate_max(pft, nit, cidx=None, cfeat=None, sign=-1, relu=False):
    """pft [B,N,C]; nit [B,M,K]; cidx [B,M] or cfeat [B,M,C] -> out [B,M,C]."""
    pft, nit = _f32(pft), _i32a(nit)
    B, N, C = pft.shape
    M, K = nit.shape[1], nit.shape[2]
    ci = None if cidx is None else _i32a(cidx)
    cf = None if cfeat is None else _f32(cfeat)
    out = np.empty((B, M, C), np.float32)
    lib().orc_aggregate_max(_ptr(pft), C, _ptr(nit), B, N, M, K, C, _ptr(ci), _ptr(cf), C, sign,
                            1 if relu else 0, _ptr(out), C)
    return out


def group_pointnet(xyz, feat, cxyz, nit):
    xyz, cxyz, nit = _f32(xyz), _f32(cxyz), _i32a(nit)
    B, N, _ = xyz.shape
    M, K = nit.shape[1], nit.shape[2]
    cf = 0 if feat is None else feat.shape[-1]
    fe = None if feat is None else _f32(feat)
    nfm = np.empty((B, M, K, 3 + cf), np.float32)
    lib().orc_group_pointnet(_ptr(xyz), _ptr(fe), cf, max(cf, 1), _ptr(cxyz), _ptr(nit), B, N, M, K, _ptr(nfm))
    return nfm


def group_offsets(xyz, feat, cidx, nit):
    xyz, cidx, nit = _f32(xyz), _i32a(cidx), _i32a(nit)
    B, N, _ = xyz.shape
    M, K = nit.shape[1], nit.shape[2]
    cf = 0 if feat is None else feat.shape[-1]
    fe = None if feat is None else _f32(feat)
    nfm = np.empty((B, M, K, 3 + cf), np.float32)
    lib().orc_group_offsets(_ptr(xyz), _ptr(fe), cf, max(cf, 1), _ptr(cidx), _ptr(nit), B, N, M, K, _ptr(nfm))
    return nfm


def group_edge(f, nit):
    f, nit = _f32(f), _i32a(nit)
    B, N, C = f.shape
    K = nit.shape[2]
    nfm = np.empty((B, N, K, 2 * C), np.float32)
    lib().orc_group_edge(_ptr(f), C, C, _ptr(nit), B, N, K, _ptr(nfm))
    return nfm


def rowgroup_max(y, G):
    """y [..., R, C] with R a multiple of G -> [..., R/G, C]."""
    y = _f32(y)
    C = y.shape[-1]
    rows = y.size // C
    assert rows % G == 0
    out = np.empty((rows // G, C), np.float32)
    lib().orc_rowgroup_max(_ptr(y), rows // G, G, C, _ptr(out), C)
    return out.reshape(y.shape[:-2] + (y.shape[-2] // G, C))


def interpolate3(xyz_dst, xyz_src, f_src):
    xyz_dst, xyz_src, f_src = _f32(xyz_dst), _f32(xyz_src), _f32(f_src)
    B, Nd, _ = xyz_dst.shape
    Ns = xyz_src.shape[1]
    C = f_src.shape[-1]
    out = np.empty((B, Nd, C), np.float32)
    lib().orc_interpolate3(_ptr(xyz_dst), _ptr(xyz_src), _ptr(f_src), C, B, Nd, Ns, C, _ptr(out), C)
    return out

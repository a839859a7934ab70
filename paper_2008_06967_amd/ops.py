"""torch.Tensor wrappers over the C ABI (argument marshalling only).

Every function allocates its outputs with ``torch.empty`` on the input's
device (unless ``out=`` is given), passes raw device pointers, leading
dimensions and the current HIP stream, and raises on a non-zero status.
All arithmetic happens in libmesorasi.so.
"""
from __future__ import annotations

import ctypes
import math

import torch

from . import _lib
from ._lib import F32, BF16, check

_vp = ctypes.c_void_p


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def _ptr(t) -> int | None:
    return None if t is None else t.data_ptr()


def _rows(t: torch.Tensor, width: int | None = None):
    """(pointer, leading dimension) of a [..., rows, C] tensor whose last dim
    is contiguous and whose leading dims collapse to one row index."""
    assert t.stride(-1) == 1, "last dimension must be contiguous"
    ld = t.stride(-2) if t.dim() >= 2 else t.shape[-1]
    # all leading dims must be row-contiguous multiples of ld
    expect = ld * t.shape[-2] if t.dim() >= 2 else None
    for d in range(t.dim() - 3, -1, -1):
        # the stride of a size-1 dimension is never used
        assert t.shape[d] == 1 or t.stride(d) == expect, "leading dimensions must collapse into rows"
        expect *= t.shape[d]
    if width is not None:
        assert t.shape[-1] >= width
    return t.data_ptr(), ld


def _check_xyz(x: torch.Tensor, name: str):
    assert x.dtype == torch.float32 and x.is_contiguous() and x.dim() == 3 and x.shape[-1] == 3, \
        f"{name} must be a contiguous float32 [B, N, 3] tensor"


def fps_workspace_bytes(B: int, N: int, M: int) -> int:
    return int(_lib.lib().mesorasi_fps_workspace(B, N, M))


def fps(xyz: torch.Tensor, M: int, want_xyz: bool = True, out_idx: torch.Tensor | None = None,
        out_xyz: torch.Tensor | None = None, ws: torch.Tensor | None = None):
    """ws: a uint8 device tensor of at least fps_workspace_bytes(B, N, M)
    (allocated here when needed and not given); its first 4 bytes read 0
    after the call unless a workgroup gave up waiting (see the C header)."""
    _check_xyz(xyz, "xyz")
    B, N, _ = xyz.shape
    idx = out_idx if out_idx is not None else torch.empty((B, M), dtype=torch.int32, device=xyz.device)
    cxyz = out_xyz if out_xyz is not None else (
        torch.empty((B, M, 3), dtype=torch.float32, device=xyz.device) if want_xyz else None)
    need = fps_workspace_bytes(B, N, M)
    if need and (ws is None or ws.numel() < need):
        ws = torch.empty(need, dtype=torch.uint8, device=xyz.device)
    wp, wn = (ws.data_ptr(), ws.numel()) if need else (None, 0)
    check(_lib.lib().mesorasi_fps(xyz.data_ptr(), B, N, M, idx.data_ptr(), _ptr(cxyz), wp, wn, _stream()), "fps")
    return idx, cxyz


def fps_prefix(idx_prev: torch.Tensor, cxyz_prev: torch.Tensor | None, M: int, out_idx: torch.Tensor | None = None,
               out_xyz: torch.Tensor | None = None, want_xyz: bool = True):
    """The sampling of M points from (idx_prev, cxyz_prev), an earlier
    fps() (or fps_prefix()) output: its first M points (see the C header)."""
    if idx_prev.dtype != torch.int32 or idx_prev.dim() != 2 or not idx_prev.is_contiguous():
        raise ValueError("idx_prev must be a contiguous [B, M_prev] int32 tensor")
    B, Mp = idx_prev.shape
    if cxyz_prev is not None:
        _check_xyz(cxyz_prev, "cxyz_prev")
        if tuple(cxyz_prev.shape[:2]) != (B, Mp):
            raise ValueError("cxyz_prev must be [B, M_prev, 3]")
    idx = out_idx if out_idx is not None else torch.empty((B, M), dtype=torch.int32, device=idx_prev.device)
    cxyz = out_xyz if out_xyz is not None else (
        torch.empty((B, M, 3), dtype=torch.float32, device=idx_prev.device)
        if want_xyz and cxyz_prev is not None else None)
    check(_lib.lib().mesorasi_fps_prefix(idx_prev.data_ptr(), _ptr(cxyz_prev), B, Mp, M, idx.data_ptr(), _ptr(cxyz),
                                         _stream()), "fps_prefix")
    return idx, cxyz


def fps_prefix_levels(idx0: torch.Tensor, cxyz0: torch.Tensor | None, Ms, out_idx=None, out_xyz=None):
    """Nested levels of M[v] points each, all prefixes of (idx0, cxyz0), in
    one launch (mesorasi_fps_prefix_levels).  Returns [(idx, cxyz)] per
    level."""
    if idx0.dtype != torch.int32 or idx0.dim() != 2 or not idx0.is_contiguous():
        raise ValueError("idx0 must be a contiguous [B, M0] int32 tensor")
    B, M0 = idx0.shape
    if cxyz0 is not None:
        _check_xyz(cxyz0, "cxyz0")
    n = len(Ms)
    idx = list(out_idx) if out_idx is not None else [
        torch.empty((B, m), dtype=torch.int32, device=idx0.device) for m in Ms]
    xyz = list(out_xyz) if out_xyz is not None else (
        [torch.empty((B, m, 3), dtype=torch.float32, device=idx0.device) for m in Ms] if cxyz0 is not None
        else [None] * n)
    Mc = (ctypes.c_int64 * max(n, 1))(*Ms)
    ic = (_vp * max(n, 1))(*[t.data_ptr() for t in idx])
    xc = (_vp * max(n, 1))(*[None if t is None else t.data_ptr() for t in xyz])
    check(_lib.lib().mesorasi_fps_prefix_levels(idx0.data_ptr(), _ptr(cxyz0), B, M0, n, ctypes.cast(Mc, _vp),
                                                ctypes.cast(ic, _vp), ctypes.cast(xc, _vp), _stream()),
          "fps_prefix_levels")
    return list(zip(idx, xyz))


def ball_query_workspace_bytes(B: int, N: int, M: int) -> int:
    return int(_lib.lib().mesorasi_ball_query_workspace(B, N, M))


def ball_query(xyz: torch.Tensor, qxyz: torch.Tensor, radius: float, K: int, want_cnt: bool = False,
               out: torch.Tensor | None = None, ws: torch.Tensor | None = None):
    """ws: a uint8 device tensor of at least ball_query_workspace_bytes(B, N,
    M) (allocated here when needed and not given)."""
    _check_xyz(xyz, "xyz")
    _check_xyz(qxyz, "qxyz")
    B, N, _ = xyz.shape
    M = qxyz.shape[1]
    nit = out if out is not None else torch.empty((B, M, K), dtype=torch.int32, device=xyz.device)
    cnt = torch.empty((B, M), dtype=torch.int32, device=xyz.device) if want_cnt else None
    need = ball_query_workspace_bytes(B, N, M)
    if need and (ws is None or ws.numel() < need):
        ws = torch.empty(need, dtype=torch.uint8, device=xyz.device)
    wp, wn = (ws.data_ptr(), ws.numel()) if need else (None, 0)
    check(_lib.lib().mesorasi_ball_query(xyz.data_ptr(), qxyz.data_ptr(), B, N, M, float(radius), K, nit.data_ptr(),
                                         _ptr(cnt), wp, wn, _stream()), "ball_query")
    return nit, cnt


def ball_query_grid_workspace_bytes(B: int, N: int) -> int:
    return int(_lib.lib().mesorasi_ball_query_grid_workspace(B, N))


def ball_query_grid_build(xyz: torch.Tensor, radius: float, ws: torch.Tensor | None = None) -> torch.Tensor:
    """Bin the clouds of xyz for ball queries of radius up to `radius`
    (mesorasi_ball_query_grid_build); returns the workspace holding the grid."""
    _check_xyz(xyz, "xyz")
    B, N, _ = xyz.shape
    need = ball_query_grid_workspace_bytes(B, N)
    if ws is None or ws.numel() < need:
        ws = torch.empty(max(need, 256), dtype=torch.uint8, device=xyz.device)
    check(_lib.lib().mesorasi_ball_query_grid_build(xyz.data_ptr(), B, N, float(radius), ws.data_ptr(), ws.numel(),
                                                    _stream()), "ball_query_grid_build")
    return ws


def ball_query_grid(xyz: torch.Tensor, qxyz: torch.Tensor, radius: float, K: int, grid: torch.Tensor,
                    want_cnt: bool = False, out: torch.Tensor | None = None):
    """ball_query() against a grid from ball_query_grid_build() on the same
    xyz (mesorasi_ball_query_grid): the same result."""
    _check_xyz(xyz, "xyz")
    _check_xyz(qxyz, "qxyz")
    B, N, _ = xyz.shape
    M = qxyz.shape[1]
    nit = out if out is not None else torch.empty((B, M, K), dtype=torch.int32, device=xyz.device)
    cnt = torch.empty((B, M), dtype=torch.int32, device=xyz.device) if want_cnt else None
    check(_lib.lib().mesorasi_ball_query_grid(xyz.data_ptr(), qxyz.data_ptr(), B, N, M, float(radius), K,
                                              nit.data_ptr(), _ptr(cnt), grid.data_ptr(), grid.numel(), _stream()),
          "ball_query_grid")
    return nit, cnt


def knn(ref: torch.Tensor, query: torch.Tensor, K: int, want_dist: bool = False, out: torch.Tensor | None = None):
    """ref [B, N, >=C], query [B, M, >=C] (last dim contiguous, may be
    column slices of wider tensors); C = ref.shape[-1]."""
    assert ref.dtype == torch.float32 and query.dtype == torch.float32
    B, N, C = ref.shape
    M = query.shape[1]
    pr, ldr = _rows(ref)
    pq, ldq = _rows(query)
    nit = out if out is not None else torch.empty((B, M, K), dtype=torch.int32, device=ref.device)
    dist = torch.empty((B, M, K), dtype=torch.float32, device=ref.device) if want_dist else None
    check(_lib.lib().mesorasi_knn(pr, ldr, pq, ldq, B, N, M, C, K, nit.data_ptr(), _ptr(dist), _stream()), "knn")
    return nit, dist


class MLPParams:
    """Weights of one shared MLP on the device, plus the host pointer arrays
    the ABI takes.  W[l] is [C_out, C_in] (torch Linear layout)."""

    def __init__(self, Ws, bs, dtype: int = F32, device="cuda"):
        self.dtype = dtype
        self.dims = [int(Ws[0].shape[1])] + [int(W.shape[0]) for W in Ws]
        self.n = len(Ws)
        self.W32 = [torch.as_tensor(W, dtype=torch.float32).to(device).contiguous() for W in Ws]
        self.b = [None if b is None else torch.as_tensor(b, dtype=torch.float32).to(device).contiguous() for b in bs]
        if dtype == BF16:
            self.W = [cast_bf16(W) for W in self.W32]
        else:
            self.W = self.W32
        self._dims_c = (ctypes.c_int32 * (self.n + 1))(*self.dims)
        self._W_c = (_vp * self.n)(*[W.data_ptr() for W in self.W])
        self._b_c = (_vp * self.n)(*[None if b is None else b.data_ptr() for b in self.b])

    @property
    def c_out(self):
        return self.dims[-1]

    def abi(self):
        return (ctypes.cast(self._dims_c, _vp), ctypes.cast(self._W_c, _vp), ctypes.cast(self._b_c, _vp))


def mlp_workspace_bytes(rows: int, p: MLPParams, pool_group: int = 0) -> int:
    d, _, _ = p.abi()
    return int(_lib.lib().mesorasi_pointwise_mlp_workspace(rows, p.n, d, p.dtype, pool_group))


def pointwise_mlp(x0: torch.Tensor, p: MLPParams, x1: torch.Tensor | None = None, relu_mask: int | None = None,
                  out_dtype: int = F32, pool_group: int = 0, out: torch.Tensor | None = None,
                  ws: torch.Tensor | None = None):
    """MLP on the rows of [x0 | x1].  x0 [..., R, c0], x1 [..., R, c1].
    pool_group > 0 returns the column max over each group of rows."""
    p0, ld0 = _rows(x0)
    c0 = x0.shape[-1]
    if x1 is not None:
        p1, ld1 = _rows(x1)
        c1 = x1.shape[-1]
    else:
        p1, ld1, c1 = None, 0, 0
    rows = math.prod(x0.shape[:-1])
    if relu_mask is None:
        relu_mask = (1 << p.n) - 1
    lead = tuple(x0.shape[:-1])
    if out is None:
        dt = torch.float32 if out_dtype == F32 else torch.bfloat16
        if pool_group:
            out = torch.empty((rows // pool_group, p.c_out), dtype=dt, device=x0.device)
        else:
            out = torch.empty(lead + (p.c_out,), dtype=dt, device=x0.device)
    py, ldy = _rows(out)
    need = mlp_workspace_bytes(rows, p, pool_group)
    if need and (ws is None or ws.numel() < need):
        ws = torch.empty(need, dtype=torch.uint8, device=x0.device)
    wp, wn = (ws.data_ptr(), ws.numel()) if need else (None, 0)
    d, W, b = p.abi()
    check(_lib.lib().mesorasi_pointwise_mlp(p0, c0, ld0, p1, c1, ld1, rows, p.n, d, W, b, relu_mask, p.dtype,
                                            out_dtype, py, ldy, pool_group, wp, wn, _stream()),
          "pointwise_mlp")
    return out


def pointwise_mlp_noalloc(x0: torch.Tensor, p: MLPParams, x1: torch.Tensor | None = None,
                          relu_mask: int | None = None, out_dtype: int = F32, pool_group: int = 0,
                          out: torch.Tensor | None = None):
    """pointwise_mlp through the allocation-free entry point: the library's
    fixed per-GPU scratch array replaces the workspace (calls that overlap
    on one GPU race).  Only `out` is allocated here, when not given."""
    p0, ld0 = _rows(x0)
    c0 = x0.shape[-1]
    if x1 is not None:
        p1, ld1 = _rows(x1)
        c1 = x1.shape[-1]
    else:
        p1, ld1, c1 = None, 0, 0
    rows = math.prod(x0.shape[:-1])
    if relu_mask is None:
        relu_mask = (1 << p.n) - 1
    if out is None:
        dt = torch.float32 if out_dtype == F32 else torch.bfloat16
        shape = (rows // pool_group, p.c_out) if pool_group else tuple(x0.shape[:-1]) + (p.c_out,)
        out = torch.empty(shape, dtype=dt, device=x0.device)
    py, ldy = _rows(out)
    d, W, b = p.abi()
    check(_lib.lib().mesorasi_pointwise_mlp_noalloc(p0, c0, ld0, p1, c1, ld1, rows, p.n, d, W, b, relu_mask,
                                                    p.dtype, out_dtype, py, ldy, pool_group, _stream()),
          "pointwise_mlp_noalloc")
    return out


def aggregate_mlp_supported(p: MLPParams, C: int) -> bool:
    """The fused aggregate-into-MLP form applies: an fp32 MLP of at least two
    layers, inputs <= 160 and outputs <= 128 channels, first layer 3 + C."""
    return (p.dtype == F32 and p.n >= 2 and p.dims[0] == 3 + C and C % 4 == 0
            and all(((d + 15) // 16) * 16 <= 160 for d in p.dims[:-1]) and all(d <= 128 for d in p.dims[1:]))


def aggregate_mlp(cxyz: torch.Tensor, pft: torch.Tensor, nit: torch.Tensor, cidx: torch.Tensor, p: MLPParams,
                  relu_mask: int | None = None, out: torch.Tensor | None = None, agg_out: torch.Tensor | None = None):
    """MLP of module i + 1 on [cxyz | module i's aggregation] with the
    aggregation done in the MLP's loader; agg_out (optional) also receives
    the aggregated rows.  cxyz [B, M, 3], pft [B, N, >=C] float32, nit
    [B, M, K], cidx [B, M]."""
    _check_xyz(cxyz, "cxyz")
    B, M, K = nit.shape
    N, C = pft.shape[1], pft.shape[-1]
    assert pft.dtype == torch.float32 and nit.is_contiguous() and cidx.is_contiguous()
    pp, ldp = _rows(pft)
    if relu_mask is None:
        relu_mask = (1 << p.n) - 1
    if out is None:
        out = torch.empty((B, M, p.c_out), dtype=torch.float32, device=pft.device)
    py, ldy = _rows(out)
    pa, lda = _rows(agg_out) if agg_out is not None else (None, 0)
    d, W, b = p.abi()
    check(_lib.lib().mesorasi_aggregate_mlp(cxyz.data_ptr(), pp, ldp, nit.data_ptr(), cidx.data_ptr(), B, N, M, K, C,
                                            p.n, d, W, b, relu_mask, py, ldy, pa, lda, _stream()), "aggregate_mlp")
    return out


def aggregate_max(pft: torch.Tensor, nit: torch.Tensor, cidx: torch.Tensor | None = None,
                  cfeat: torch.Tensor | None = None, sign: int = -1, relu: bool = False,
                  out: torch.Tensor | None = None):
    """pft [B, N, >=C] float32 or bfloat16; nit [B, M, K] int32;
    cidx [B, M] int32 or cfeat [B, M, >=C] (same dtype as pft)."""
    B, N, C = pft.shape
    M, K = nit.shape[1], nit.shape[2]
    dt = F32 if pft.dtype == torch.float32 else BF16
    pp, ldp = _rows(pft)
    if cfeat is not None:
        assert cfeat.dtype == pft.dtype
        pc, ldc = _rows(cfeat)
    else:
        pc, ldc = None, 0
    if out is None:
        out = torch.empty((B, M, C), dtype=torch.float32, device=pft.device)
    po, ldo = _rows(out)
    assert nit.is_contiguous() and nit.dtype == torch.int32
    check(_lib.lib().mesorasi_aggregate_max(pp, ldp, dt, nit.data_ptr(), B, N, M, K, C, _ptr(cidx), pc, ldc, sign,
                                            1 if relu else 0, po, ldo, _stream()), "aggregate_max")
    return out


def conventional_workspace_bytes(B: int, M: int, K: int, p: MLPParams) -> int:
    d, _, _ = p.abi()
    return int(_lib.lib().mesorasi_conventional_workspace(B, M, K, p.n, d, p.dtype))


def conventional_module(nit: torch.Tensor, p: MLPParams, xyz: torch.Tensor | None = None,
                        feat: torch.Tensor | None = None, cxyz: torch.Tensor | None = None, grouping: int = 0,
                        relu_mask: int | None = None, out: torch.Tensor | None = None,
                        ws: torch.Tensor | None = None):
    """grouping 0: [xyz_j - cxyz_c | feat_j] (PointNet++); grouping 1:
    [f_i | f_j - f_i] with f = feat (DGCNN edge features)."""
    B, M, K = nit.shape
    if grouping == 0:
        N = xyz.shape[1]
    else:
        N = feat.shape[1]
    cf = 0 if feat is None else feat.shape[-1]
    pf, ldf = _rows(feat) if feat is not None else (None, max(cf, 1))
    if relu_mask is None:
        relu_mask = (1 << p.n) - 1
    if out is None:
        out = torch.empty((B, M, p.c_out), dtype=torch.float32, device=nit.device)
    po, ldo = _rows(out)
    need = conventional_workspace_bytes(B, M, K, p)
    if ws is None or ws.numel() < need:
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device=nit.device)
    d, W, b = p.abi()
    check(_lib.lib().mesorasi_conventional_module(_ptr(xyz), pf, cf, ldf, _ptr(cxyz), nit.data_ptr(), B, N, M, K,
                                                  grouping, p.n, d, W, b, relu_mask, p.dtype, po, ldo,
                                                  ws.data_ptr(), ws.numel(), _stream()), "conventional_module")
    return out


def ltd_workspace_bytes(B: int, M: int, K: int, p: MLPParams) -> int:
    d, _, _ = p.abi()
    return int(_lib.lib().mesorasi_ltd_workspace(B, M, K, p.n, d, p.dtype))


def ltd_module(p1: torch.Tensor, q: torch.Tensor, nit: torch.Tensor, p: MLPParams, b1: torch.Tensor | None = None,
               relu_mask: int | None = None, out: torch.Tensor | None = None, ws: torch.Tensor | None = None):
    """Limited delayed aggregation (Sec. 7.3): p1 [B, N, >=C1] = the first
    layer's product on the input points, q [B, M, >=C1] = its centroid
    term, b1 [C1] the first layer's bias; p = the remaining layers.
    Returns max_k MLP_rest(ReLU(p1[nit] - q + b1)) [B, M, C_out]."""
    B, M, K = nit.shape
    N, C1 = p1.shape[1], p.dims[0]
    pp, ldp = _rows(p1, C1)
    pq, ldq = _rows(q, C1)
    if relu_mask is None:
        relu_mask = (1 << p.n) - 1
    if out is None:
        out = torch.empty((B, M, p.c_out), dtype=torch.float32, device=nit.device)
    po, ldo = _rows(out)
    need = ltd_workspace_bytes(B, M, K, p)
    if ws is None or ws.numel() < need:
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device=nit.device)
    d, W, b = p.abi()
    check(_lib.lib().mesorasi_ltd_module(pp, ldp, pq, ldq, _ptr(b1), nit.data_ptr(), B, N, M, K, C1, p.n, d, W, b,
                                         relu_mask, p.dtype, po, ldo, ws.data_ptr(), ws.numel(), _stream()),
          "ltd_module")
    return out


def interpolate3(xyz_dst: torch.Tensor, xyz_src: torch.Tensor, f_src: torch.Tensor,
                 out: torch.Tensor | None = None):
    _check_xyz(xyz_dst, "xyz_dst")
    _check_xyz(xyz_src, "xyz_src")
    B, Nd, _ = xyz_dst.shape
    Ns = xyz_src.shape[1]
    C = f_src.shape[-1]
    ps, lds = _rows(f_src)
    if out is None:
        out = torch.empty((B, Nd, C), dtype=torch.float32, device=f_src.device)
    po, ldo = _rows(out)
    check(_lib.lib().mesorasi_interpolate3(xyz_dst.data_ptr(), xyz_src.data_ptr(), ps, lds, B, Nd, Ns, C, po, ldo,
                                           _stream()), "interpolate3")
    return out


def three_nn(xyz_dst: torch.Tensor, xyz_src: torch.Tensor, out_nit: torch.Tensor | None = None,
             out_dist: torch.Tensor | None = None):
    """The 3 nearest sources of every destination (indices, squared
    distances), as mesorasi_knn with K = 3."""
    _check_xyz(xyz_dst, "xyz_dst")
    _check_xyz(xyz_src, "xyz_src")
    B, Nd, _ = xyz_dst.shape
    Ns = xyz_src.shape[1]
    nit = out_nit if out_nit is not None else torch.empty((B, Nd, 3), dtype=torch.int32, device=xyz_dst.device)
    dist = out_dist if out_dist is not None else torch.empty((B, Nd, 3), dtype=torch.float32, device=xyz_dst.device)
    check(_lib.lib().mesorasi_three_nn(xyz_dst.data_ptr(), xyz_src.data_ptr(), B, Nd, Ns, nit.data_ptr(),
                                       dist.data_ptr(), _stream()), "three_nn")
    return nit, dist


def interpolate3_apply(nit: torch.Tensor, dist: torch.Tensor, f_src: torch.Tensor, out: torch.Tensor | None = None):
    """Inverse-distance interpolation from precomputed 3-NN (three_nn)."""
    assert nit.dtype == torch.int32 and nit.is_contiguous() and dist.dtype == torch.float32 and dist.is_contiguous()
    B, Nd, _ = nit.shape
    Ns, C = f_src.shape[1], f_src.shape[-1]
    ps, lds = _rows(f_src)
    if out is None:
        out = torch.empty((B, Nd, C), dtype=torch.float32, device=f_src.device)
    po, ldo = _rows(out)
    check(_lib.lib().mesorasi_interpolate3_apply(nit.data_ptr(), dist.data_ptr(), ps, lds, B, Nd, Ns, C, po, ldo,
                                                 _stream()), "interpolate3_apply")
    return out


def interpolate3_add(nit: torch.Tensor, dist: torch.Tensor, f_src: torch.Tensor, add: torch.Tensor,
                     relu: bool = True, out: torch.Tensor | None = None):
    """phi(interpolation of f_src from precomputed 3-NN + add), phi = ReLU
    when relu: a feature-propagation first layer whose interpolated part
    was multiplied on the coarse points.  out may be add itself."""
    assert nit.dtype == torch.int32 and nit.is_contiguous() and dist.dtype == torch.float32 and dist.is_contiguous()
    B, Nd, _ = nit.shape
    Ns, C = f_src.shape[1], f_src.shape[-1]
    assert add.shape[:2] == (B, Nd) and add.shape[-1] == C and add.dtype == torch.float32
    ps, lds = _rows(f_src)
    pa, lda = _rows(add)
    if out is None:
        out = torch.empty((B, Nd, C), dtype=torch.float32, device=f_src.device)
    po, ldo = _rows(out)
    check(_lib.lib().mesorasi_interpolate3_add(nit.data_ptr(), dist.data_ptr(), ps, lds, B, Nd, Ns, C, pa, lda,
                                               1 if relu else 0, po, ldo, _stream()), "interpolate3_add")
    return out


def interpolate3_mlp_supported(p: MLPParams, rows: int) -> bool:
    """mesorasi_interpolate3_mlp applies: an fp32 MLP whose layers are all at
    most 128 wide (the register-resident MLP), first layer a multiple of 4,
    and, when the layers' permuted weights do not fit 160 KB of LDS
    together, at most one 32-row tile per wave (8 per compute unit).  This
    mirrors the library's plan."""
    if p.dtype != F32 or p.dims[0] % 4 != 0 or any(d > 128 for d in p.dims):
        return False
    h0 = ((p.dims[0] + 1) // 2 + 15) // 16 * 16     # first-layer k steps, as the library pads them
    cap, off, phases = 160 * 1024, 0, 1
    for l in range(p.n):
        nob = (p.dims[l + 1] + 31) // 32
        steps = h0 if l == 0 else 16 * ((p.dims[l] + 31) // 32)
        size = 4 * (nob * steps * 64 + nob * 32)
        if off + size > cap:
            phases, off = phases + 1, 0
        off += size
    if phases == 1:
        return True
    cus = torch.cuda.get_device_properties(torch.cuda.current_device()).multi_processor_count
    return (rows + 31) // 32 <= 8 * cus


def interpolate3_mlp(nit: torch.Tensor, dist: torch.Tensor, f_src: torch.Tensor, add: torch.Tensor, p: MLPParams,
                     relu: bool = True, relu_mask: int | None = None, out: torch.Tensor | None = None):
    """MLP on the rows phi(interpolation of f_src + add) in one kernel
    (mesorasi_interpolate3_mlp)."""
    assert nit.dtype == torch.int32 and nit.is_contiguous() and dist.dtype == torch.float32 and dist.is_contiguous()
    B, Nd, _ = nit.shape
    Ns = f_src.shape[1]
    assert add.shape[:2] == (B, Nd) and add.shape[-1] == p.dims[0] and f_src.shape[-1] == p.dims[0]
    ps, lds = _rows(f_src)
    pa, lda = _rows(add)
    if out is None:
        out = torch.empty((B, Nd, p.c_out), dtype=torch.float32, device=f_src.device)
    po, ldo = _rows(out)
    d, W, b = p.abi()
    rm = (1 << p.n) - 1 if relu_mask is None else relu_mask
    check(_lib.lib().mesorasi_interpolate3_mlp(nit.data_ptr(), dist.data_ptr(), ps, lds, B, Nd, Ns, pa, lda,
                                               1 if relu else 0, p.n, d, W, b, rm, po, ldo, _stream()),
          "interpolate3_mlp")
    return out


def cast_bf16(x: torch.Tensor) -> torch.Tensor:
    """float32 -> bfloat16 (round to nearest even) on the device."""
    assert x.dtype == torch.float32 and x.is_contiguous()
    y = torch.empty(x.shape, dtype=torch.bfloat16, device=x.device)
    check(_lib.lib().mesorasi_cast_bf16(x.data_ptr(), x.numel(), y.data_ptr(), _stream()), "cast_bf16")
    return y


def edgeconv_fold(W: torch.Tensor, b: torch.Tensor | None):
    """W [C_out, 2C] -> ([W1 - W2 ; W2] [2 C_out, C], [b ; 0])."""
    Cout, C2 = W.shape
    C = C2 // 2
    Wo = torch.empty((2 * Cout, C), dtype=torch.float32, device=W.device)
    bo = torch.empty((2 * Cout,), dtype=torch.float32, device=W.device)
    check(_lib.lib().mesorasi_edgeconv_fold(W.data_ptr(), _ptr(b), C, Cout, Wo.data_ptr(), bo.data_ptr(), _stream()),
          "edgeconv_fold")
    return Wo, bo


def count_out_of_range(idx: torch.Tensor, bound: int, out: torch.Tensor | None = None) -> torch.Tensor:
    """Device int32 scalar: entries of idx outside [0, bound) (debug check)."""
    assert idx.dtype == torch.int32 and idx.is_contiguous()
    count = out if out is not None else torch.empty((), dtype=torch.int32, device=idx.device)
    check(_lib.lib().mesorasi_count_out_of_range(idx.data_ptr(), idx.numel(), int(bound), count.data_ptr(),
                                                 _stream()), "count_out_of_range")
    return count

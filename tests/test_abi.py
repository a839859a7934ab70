"""Host-side checks of the C ABI that need no GPU: the library loads, it
exports every entry point include/mesorasi.h declares, and argument
validation returns the documented status before any HIP call is made."""
import ctypes
import os
import re

import pytest

from paper_2008_06967_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mesorasi.h")

NULL = None
FAKE = ctypes.c_void_p(0x1000)   # never dereferenced: every call below fails validation first


def declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(mesorasi_\w+)\s*\(", src)))


def test_every_declared_symbol_is_exported_and_bound():
    L = _lib.lib()
    names = declared()
    assert len(names) >= 14
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(_lib.SIGNATURES)


def test_version_and_strings():
    L = _lib.lib()
    assert L.mesorasi_version() == 1
    assert L.mesorasi_strerror(0) == b"ok"
    assert L.mesorasi_strerror(-1) == b"invalid argument"
    assert L.mesorasi_strerror(-4) == b"workspace too small"


def st(fn, *args):
    return getattr(_lib.lib(), fn)(*args)


def test_fps_validation():
    f = "mesorasi_fps"
    assert st(f, FAKE, 1, 10, 11, FAKE, NULL, NULL, 0, NULL) == _lib.EINVAL          # M > N
    assert st(f, FAKE, -1, 10, 5, FAKE, NULL, NULL, 0, NULL) == _lib.EINVAL          # B < 0
    assert st(f, NULL, 1, 10, 5, FAKE, NULL, NULL, 0, NULL) == _lib.EINVAL           # NULL xyz
    assert st(f, FAKE, 1, 70000, 5, FAKE, NULL, NULL, 0, NULL) == _lib.EUNSUPPORTED  # N too large
    assert st(f, NULL, 0, 10, 5, NULL, NULL, NULL, 0, NULL) == _lib.OK               # empty batch
    st(f, FAKE, 1, 10, 11, FAKE, NULL, NULL, 0, NULL)
    assert b"M = 11" in _lib.lib().mesorasi_last_error()


def test_fps_prefix_validation():
    f = "mesorasi_fps_prefix"
    assert st(f, FAKE, FAKE, 1, 10, 11, FAKE, FAKE, NULL) == _lib.EINVAL          # M > M_prev
    assert st(f, FAKE, FAKE, -1, 10, 5, FAKE, FAKE, NULL) == _lib.EINVAL          # B < 0
    assert st(f, NULL, FAKE, 1, 10, 5, FAKE, FAKE, NULL) == _lib.EINVAL           # NULL idx_prev
    assert st(f, FAKE, FAKE, 1, 10, 5, NULL, FAKE, NULL) == _lib.EINVAL           # NULL idx
    assert st(f, FAKE, NULL, 1, 10, 5, FAKE, FAKE, NULL) == _lib.EINVAL           # cxyz without cxyz_prev
    assert st(f, FAKE, FAKE, 1, 70000, 5, FAKE, FAKE, NULL) == _lib.EUNSUPPORTED  # M_prev too large
    assert st(f, NULL, NULL, 0, 10, 5, NULL, NULL, NULL) == _lib.OK               # empty batch
    assert st(f, NULL, NULL, 3, 10, 0, NULL, NULL, NULL) == _lib.OK               # nothing to select
    st(f, FAKE, FAKE, 1, 10, 11, FAKE, FAKE, NULL)
    assert b"M_prev = 10" in _lib.lib().mesorasi_last_error()


def test_fps_prefix_levels_validation():
    f = "mesorasi_fps_prefix_levels"
    M = (ctypes.c_int64 * 2)(5, 11)
    P = (ctypes.c_void_p * 2)(0x1000, 0x2000)
    assert st(f, FAKE, FAKE, 1, 10, 2, M, P, P, NULL) == _lib.EINVAL        # M[1] > M0
    assert st(f, FAKE, FAKE, -1, 10, 2, M, P, P, NULL) == _lib.EINVAL       # B < 0
    assert st(f, FAKE, FAKE, 1, 10, 9, M, P, P, NULL) == _lib.EINVAL        # too many levels
    assert st(f, FAKE, FAKE, 1, 10, 2, NULL, P, P, NULL) == _lib.EINVAL     # NULL M
    M2 = (ctypes.c_int64 * 2)(5, 3)
    assert st(f, NULL, FAKE, 1, 10, 2, M2, P, P, NULL) == _lib.EINVAL       # NULL idx0
    assert st(f, FAKE, NULL, 1, 10, 2, M2, P, P, NULL) == _lib.EINVAL       # cxyz without cxyz0
    assert st(f, FAKE, FAKE, 1, 70000, 2, M2, P, P, NULL) == _lib.EUNSUPPORTED
    assert st(f, NULL, NULL, 0, 10, 2, M2, P, P, NULL) == _lib.OK           # empty batch
    assert st(f, NULL, NULL, 3, 10, 0, NULL, NULL, NULL, NULL) == _lib.OK   # no levels
    st(f, FAKE, FAKE, 1, 10, 2, M, P, P, NULL)
    assert b"M[1] = 11" in _lib.lib().mesorasi_last_error()


def test_ball_query_grid_validation():
    f, b = "mesorasi_ball_query_grid", "mesorasi_ball_query_grid_build"
    L = _lib.lib()
    need = L.mesorasi_ball_query_grid_workspace(2, 4096)
    assert need > 2 * 4096 * 16
    assert L.mesorasi_ball_query_grid_workspace(2, 70000) == 0
    assert st(b, FAKE, -1, 10, 0.1, FAKE, 1 << 20, NULL) == _lib.EINVAL            # B < 0
    assert st(b, FAKE, 1, 10, 0.0, FAKE, 1 << 20, NULL) == _lib.EINVAL             # radius 0
    assert st(b, NULL, 1, 10, 0.1, FAKE, 1 << 20, NULL) == _lib.EINVAL             # NULL xyz
    assert st(b, FAKE, 1, 10, 0.1, NULL, 1 << 20, NULL) == _lib.EWORKSPACE         # NULL ws
    assert st(b, FAKE, 1, 10, 0.1, FAKE, 16, NULL) == _lib.EWORKSPACE              # too small
    assert st(b, FAKE, 1, 70000, 0.1, FAKE, 1 << 30, NULL) == _lib.EUNSUPPORTED
    assert st(b, NULL, 0, 10, 0.1, NULL, 0, NULL) == _lib.OK                      # empty batch
    assert st(f, FAKE, FAKE, 1, 10, 5, 0.1, 0, FAKE, NULL, FAKE, 1 << 20, NULL) == _lib.EINVAL      # K = 0
    assert st(f, FAKE, FAKE, 1, 10, 5, 0.1, 2000, FAKE, NULL, FAKE, 1 << 20, NULL) == _lib.EUNSUPPORTED
    assert st(f, FAKE, FAKE, 1, 0, 5, 0.1, 8, FAKE, NULL, FAKE, 1 << 20, NULL) == _lib.EINVAL       # N = 0, M > 0
    assert st(f, FAKE, FAKE, 1, 10, 5, 0.1, 8, FAKE, NULL, NULL, 1 << 20, NULL) == _lib.EWORKSPACE  # no grid
    assert st(f, FAKE, FAKE, 1, 10, 5, 0.1, 8, FAKE, NULL, FAKE, 16, NULL) == _lib.EWORKSPACE
    assert st(f, NULL, NULL, 0, 10, 5, 0.1, 8, NULL, NULL, NULL, 0, NULL) == _lib.OK                # empty batch


def test_fps_workspace():
    """Small clouds run one workgroup per cloud and need no workspace; large
    ones exchange winners through one, which must be big enough and 8-byte
    aligned."""
    L = _lib.lib()
    f = "mesorasi_fps"
    assert L.mesorasi_fps_workspace(32, 1024, 512) == 0
    assert L.mesorasi_fps_workspace(4, 16384, 4096) == 0
    need = L.mesorasi_fps_workspace(4, 40000, 4096)
    assert need > 0 and need % 8 == 0
    assert L.mesorasi_fps_workspace(8, 40000, 4096) > need                           # grows with the batch
    assert L.mesorasi_fps_workspace(4, 40000, 1) == 0                                # nothing to exchange
    assert L.mesorasi_fps_workspace(4, 100, 200) == 0                                # invalid sizes
    assert st(f, FAKE, 4, 40000, 4096, FAKE, NULL, NULL, 0, NULL) == _lib.EWORKSPACE
    assert st(f, FAKE, 4, 40000, 4096, FAKE, NULL, FAKE, need - 8, NULL) == _lib.EWORKSPACE
    assert st(f, FAKE, 4, 40000, 4096, FAKE, NULL, ctypes.c_void_p(0x1004), need, NULL) == _lib.EINVAL
    assert b"aligned" in L.mesorasi_last_error()


def test_ball_query_validation():
    f = "mesorasi_ball_query"
    z = (NULL, 0, NULL)        # ws, ws_bytes, stream
    assert st(f, FAKE, FAKE, 1, 10, 5, 0.2, 0, FAKE, NULL, *z) == _lib.EINVAL              # K < 1
    assert st(f, FAKE, FAKE, 1, 10, 5, -0.2, 4, FAKE, NULL, *z) == _lib.EINVAL             # radius <= 0
    assert st(f, FAKE, FAKE, 1, 10, 5, float("nan"), 4, FAKE, NULL, *z) == _lib.EINVAL
    assert st(f, FAKE, FAKE, 1, 10, 5, float("inf"), 4, FAKE, NULL, *z) == _lib.EINVAL
    assert st(f, FAKE, FAKE, 1, 10, 5, 0.2, 2000, FAKE, NULL, *z) == _lib.EUNSUPPORTED
    assert st(f, FAKE, FAKE, 1, 0, 5, 0.2, 4, FAKE, NULL, *z) == _lib.EINVAL               # N = 0 < M
    assert st(f, NULL, FAKE, 1, 10, 5, 0.2, 4, FAKE, NULL, *z) == _lib.EINVAL
    assert st(f, NULL, NULL, 1, 10, 0, 0.2, 4, NULL, NULL, *z) == _lib.OK                  # M = 0


def test_ball_query_workspace():
    """Clouds of 8192 points or more are binned into a grid in a workspace,
    which must be large enough and 256-byte aligned."""
    L = _lib.lib()
    f = "mesorasi_ball_query"
    assert L.mesorasi_ball_query_workspace(32, 1024, 512) == 0
    need = L.mesorasi_ball_query_workspace(4, 16384, 4096)
    assert need > 4 * 16384 * 16
    assert L.mesorasi_ball_query_workspace(8, 16384, 4096) > need
    assert L.mesorasi_ball_query_workspace(4, 16384, 0) == 0
    assert st(f, FAKE, FAKE, 4, 16384, 4096, 0.1, 64, FAKE, NULL, NULL, 0, NULL) == _lib.EWORKSPACE
    assert st(f, FAKE, FAKE, 4, 16384, 4096, 0.1, 64, FAKE, NULL, FAKE, need - 1, NULL) == _lib.EWORKSPACE
    assert st(f, FAKE, FAKE, 4, 16384, 4096, 0.1, 64, FAKE, NULL, ctypes.c_void_p(0x1080), need, NULL) == _lib.EINVAL
    assert b"aligned" in L.mesorasi_last_error()


def test_knn_validation():
    f = "mesorasi_knn"
    assert st(f, FAKE, 3, FAKE, 3, 1, 10, 10, 3, 11, FAKE, NULL, NULL) == _lib.EINVAL        # K > N
    assert st(f, FAKE, 2, FAKE, 3, 1, 10, 10, 3, 4, FAKE, NULL, NULL) == _lib.EINVAL         # ld < C
    assert st(f, FAKE, 3, FAKE, 3, 1, 100, 10, 3, 65, FAKE, NULL, NULL) == _lib.EUNSUPPORTED # K > 64
    assert st(f, FAKE, 300, FAKE, 300, 1, 100, 10, 300, 4, FAKE, NULL, NULL) == _lib.EUNSUPPORTED  # C > 128
    assert st(f, FAKE, 3, FAKE, 3, 1, 10, 10, 0, 4, FAKE, NULL, NULL) == _lib.EINVAL         # C < 1


def _mlp_args(dims):
    d = (ctypes.c_int32 * len(dims))(*dims)
    W = (ctypes.c_void_p * (len(dims) - 1))(*([0x1000] * (len(dims) - 1)))
    b = (ctypes.c_void_p * (len(dims) - 1))()
    return ctypes.cast(d, ctypes.c_void_p), ctypes.cast(W, ctypes.c_void_p), ctypes.cast(b, ctypes.c_void_p)


def test_mlp_validation_and_workspace():
    L = _lib.lib()
    d, W, b = _mlp_args([3, 64, 64, 128])
    f = "mesorasi_pointwise_mlp"
    # dims[0] != c0 + c1
    assert st(f, FAKE, 4, 4, NULL, 0, 0, 10, 3, d, W, b, 7, 0, 0, FAKE, 128, 0, NULL, 0, NULL) == _lib.EINVAL
    # pooling without final ReLU
    assert st(f, FAKE, 3, 3, NULL, 0, 0, 10, 3, d, W, b, 3, 0, 0, FAKE, 128, 5, FAKE, 1 << 20, NULL) == \
        _lib.EUNSUPPORTED
    # rows % pool_group
    assert st(f, FAKE, 3, 3, NULL, 0, 0, 10, 3, d, W, b, 7, 0, 0, FAKE, 128, 3, FAKE, 1 << 20, NULL) == _lib.EINVAL
    # pool groups are limited to 2^31 - 1 rows
    assert st(f, FAKE, 3, 3, NULL, 0, 0, 1 << 32, 3, d, W, b, 7, 0, 0, FAKE, 128, 1 << 32, FAKE, 1 << 20, NULL) == \
        _lib.EUNSUPPORTED
    # narrow fp32 MLPs run fused and need no workspace; wide ones run layer by layer
    assert L.mesorasi_pointwise_mlp_workspace(10, 3, d, 0, 0) == 0
    dw, Ww, bw = _mlp_args([3, 200, 200, 256])
    need = L.mesorasi_pointwise_mlp_workspace(10, 3, dw, 0, 0)
    assert need > 0
    assert st(f, FAKE, 3, 3, NULL, 0, 0, 10, 3, dw, Ww, bw, 7, 0, 0, FAKE, 256, 0, FAKE, need - 1, NULL) == \
        _lib.EWORKSPACE
    # ld_y < width
    assert st(f, FAKE, 3, 3, NULL, 0, 0, 10, 3, d, W, b, 7, 0, 0, FAKE, 64, 0, FAKE, need, NULL) == _lib.EINVAL
    # too many layers
    d9, W9, b9 = _mlp_args([4] * 10)
    assert st(f, FAKE, 4, 4, NULL, 0, 0, 10, 9, d9, W9, b9, 0, 0, 0, FAKE, 4, 0, NULL, 0, NULL) == \
        _lib.EUNSUPPORTED
    # one layer needs no workspace; two need one buffer, three need two
    d1, _, _ = _mlp_args([3, 8])
    assert L.mesorasi_pointwise_mlp_workspace(100, 1, d1, 0, 0) == 0
    d2, _, _ = _mlp_args([3, 200, 200])
    d3, _, _ = _mlp_args([3, 200, 200, 200])
    one = L.mesorasi_pointwise_mlp_workspace(1000, 2, d2, 0, 0)
    # (includes split-K partial sums when the tile grid is small)
    assert one >= 1000 * 200 * 4 and L.mesorasi_pointwise_mlp_workspace(1000, 3, d3, 0, 0) >= one + 1000 * 200 * 4
    assert L.mesorasi_pointwise_mlp_workspace(1000, 2, d2, 1, 0) < one   # bf16 activations are half the size
    assert st(f, NULL, 3, 3, NULL, 0, 0, 0, 3, d, W, b, 7, 0, 0, NULL, 128, 0, NULL, 0, NULL) == _lib.OK  # rows = 0


def test_mlp_noalloc_validation():
    """The allocation-free MLP checks its arguments like the workspace form
    and refuses work beyond its fixed scratch array, before any HIP call."""
    L = _lib.lib()
    f = "mesorasi_pointwise_mlp_noalloc"
    d, W, b = _mlp_args([3, 64, 64, 128])
    assert st(f, FAKE, 4, 4, NULL, 0, 0, 10, 3, d, W, b, 7, 0, 0, FAKE, 128, 0, NULL) == _lib.EINVAL   # dims[0]
    assert st(f, FAKE, 3, 3, NULL, 0, 0, 10, 3, d, W, b, 7, 0, 0, FAKE, 128, 3, NULL) == _lib.EINVAL   # rows % G
    assert st(f, NULL, 3, 3, NULL, 0, 0, 0, 3, d, W, b, 7, 0, 0, NULL, 128, 0, NULL) == _lib.OK        # rows = 0
    dw, Ww, bw = _mlp_args([3, 200, 200, 256])
    rows = 1 << 20
    assert L.mesorasi_pointwise_mlp_workspace(rows, 3, dw, 0, 0) > _lib.NOALLOC_WS_BYTES
    assert st(f, FAKE, 3, 3, NULL, 0, 0, rows, 3, dw, Ww, bw, 7, 0, 0, FAKE, 256, 0, NULL) == _lib.EUNSUPPORTED
    assert b"scratch" in L.mesorasi_last_error()
    m = re.search(r"#define MESORASI_NOALLOC_WS_BYTES \((\d+)u << (\d+)\)", open(HEADER).read())
    assert m and int(m.group(1)) << int(m.group(2)) == _lib.NOALLOC_WS_BYTES


def test_aggregate_validation():
    f = "mesorasi_aggregate_max"
    assert st(f, FAKE, 64, 0, FAKE, 1, 10, 5, 4, 64, FAKE, FAKE, 64, -1, 0, FAKE, 64, NULL) == _lib.EINVAL  # both
    assert st(f, FAKE, 64, 0, FAKE, 1, 10, 5, 4, 64, NULL, NULL, 0, 2, 0, FAKE, 64, NULL) == _lib.EINVAL    # sign
    assert st(f, FAKE, 32, 0, FAKE, 1, 10, 5, 4, 64, NULL, NULL, 0, -1, 0, FAKE, 64, NULL) == _lib.EINVAL   # ld
    assert st(f, FAKE, 64, 7, FAKE, 1, 10, 5, 4, 64, NULL, NULL, 0, -1, 0, FAKE, 64, NULL) == \
        _lib.EUNSUPPORTED                                                                                  # dtype
    assert st(f, NULL, 64, 0, FAKE, 1, 10, 5, 4, 64, NULL, NULL, 0, -1, 0, FAKE, 64, NULL) == _lib.EINVAL


def test_conventional_validation_and_workspace():
    L = _lib.lib()
    d, W, b = _mlp_args([3, 64, 64, 128])
    f = "mesorasi_conventional_module"
    # grouping 1 needs M == N
    assert st(f, NULL, FAKE, 3, 3, NULL, FAKE, 1, 10, 5, 4, 1, 3, d, W, b, 7, 0, FAKE, 128, FAKE, 1 << 30,
              NULL) == _lib.EINVAL
    # dims[0] inconsistent with grouping 0 and cf = 2
    assert st(f, FAKE, FAKE, 2, 2, FAKE, FAKE, 1, 10, 5, 4, 0, 3, d, W, b, 7, 0, FAKE, 128, FAKE, 1 << 30,
              NULL) == _lib.EINVAL
    need = L.mesorasi_conventional_workspace(1, 5, 4, 3, d, 0)
    assert need >= 5 * 4 * 3 * 4
    assert st(f, FAKE, NULL, 0, 1, FAKE, FAKE, 1, 10, 5, 4, 0, 3, d, W, b, 7, 0, FAKE, 128, FAKE, need - 1,
              NULL) == _lib.EWORKSPACE
    assert st(f, FAKE, NULL, 0, 1, FAKE, FAKE, 1, 10, 5, 4, 0, 3, d, W, b, 3, 0, FAKE, 128, FAKE, need,
              NULL) == _lib.EUNSUPPORTED   # last layer without ReLU


def test_ltd_validation_and_workspace():
    L = _lib.lib()
    d, W, b = _mlp_args([64, 64, 128])          # the remaining layers after the hoisted first one
    f = "mesorasi_ltd_module"
    args = lambda C1, n, ld_p, ws, relu=3, ws_ptr=FAKE: (FAKE, ld_p, FAKE, 64, NULL, FAKE, 1, 10, 5, 4, C1, n, d, W, b,
                                                        relu, 0, FAKE, 128, ws_ptr, ws, NULL)
    need = L.mesorasi_ltd_workspace(1, 5, 4, 2, d, 0)
    assert need >= 5 * 4 * 64 * 4                                             # the first-layer rows
    assert st(f, *args(64, 2, 64, need - 1)) == _lib.EWORKSPACE
    assert st(f, *args(32, 2, 64, need)) == _lib.EINVAL                      # dims[0] != C1
    assert st(f, *args(64, 2, 32, need)) == _lib.EINVAL                      # ld_p < C1
    assert st(f, *args(64, 0, 64, need)) == _lib.EUNSUPPORTED                # no remaining layer
    assert st(f, *args(64, 2, 64, need, relu=1)) == _lib.EUNSUPPORTED        # last layer without ReLU
    assert L.mesorasi_ltd_workspace(1, 5, 4, 0, d, 0) == 0


def test_misc_validation():
    assert st("mesorasi_interpolate3", FAKE, FAKE, FAKE, 8, 1, 10, 2, 8, FAKE, 8, NULL) == _lib.EINVAL  # Ns < 3
    assert st("mesorasi_cast_bf16", FAKE, -1, FAKE, NULL) == _lib.EINVAL
    assert st("mesorasi_cast_bf16", NULL, 0, NULL, NULL) == _lib.OK
    assert st("mesorasi_edgeconv_fold", FAKE, NULL, 0, 4, FAKE, FAKE, NULL) == _lib.EINVAL


def test_product_path_does_not_touch_the_oracle():
    """The HIP path's sources never import, load or name the oracle."""
    pkg = os.path.join(ROOT, "paper_2008_06967_amd")
    for dirpath, _, files in os.walk(pkg):
        for fn in files:
            if fn.endswith((".py", ".hip", ".h", ".cpp")):
                src = open(os.path.join(dirpath, fn)).read()
                assert "import oracle" not in src and "from oracle" not in src and "liboracle" not in src, fn


def test_three_nn_and_apply_validation():
    assert st("mesorasi_three_nn", FAKE, FAKE, 1, 10, 2, FAKE, FAKE, NULL) == _lib.EINVAL         # Ns < 3
    assert st("mesorasi_three_nn", FAKE, NULL, 1, 10, 5, FAKE, FAKE, NULL) == _lib.EINVAL         # NULL src
    assert st("mesorasi_three_nn", NULL, NULL, 0, 10, 5, NULL, NULL, NULL) == _lib.OK             # empty batch
    f = "mesorasi_interpolate3_apply"
    assert st(f, FAKE, FAKE, FAKE, 4, 1, 10, 5, 8, FAKE, 8, NULL) == _lib.EINVAL                  # ld_src < C
    assert st(f, FAKE, NULL, FAKE, 8, 1, 10, 5, 8, FAKE, 8, NULL) == _lib.EINVAL                  # NULL dist
    assert st(f, FAKE, FAKE, FAKE, 8, 1, 10, 0, 8, FAKE, 8, NULL) == _lib.EINVAL                  # Ns = 0
    assert st(f, NULL, NULL, NULL, 8, 1, 0, 5, 8, NULL, 8, NULL) == _lib.OK                       # Nd = 0


def test_interpolate3_add_validation():
    f = "mesorasi_interpolate3_add"
    A = ctypes.c_void_p(0x2000)                     # another buffer (never dereferenced either)
    assert st(f, FAKE, FAKE, FAKE, 8, 1, 10, 5, 8, A, 4, 1, FAKE, 8, NULL) == _lib.EINVAL          # ld_add < C
    assert st(f, FAKE, FAKE, FAKE, 8, 1, 10, 5, 8, NULL, 8, 1, FAKE, 8, NULL) == _lib.EINVAL        # NULL add
    assert st(f, FAKE, FAKE, FAKE, 8, 1, 10, 5, 8, FAKE, 12, 1, FAKE, 8, NULL) == _lib.EINVAL      # aliased, other ld
    assert st(f, FAKE, FAKE, FAKE, 8, 1, 10, 0, 8, A, 8, 1, FAKE, 8, NULL) == _lib.EINVAL          # Ns = 0
    assert st(f, NULL, NULL, NULL, 8, 1, 0, 5, 8, NULL, 8, 1, NULL, 8, NULL) == _lib.OK            # Nd = 0


def test_interpolate3_mlp_validation():
    f = "mesorasi_interpolate3_mlp"
    A = ctypes.c_void_p(0x2000)
    d, W, b = _mlp_args([128, 128, 128])
    args = lambda **k: [FAKE, FAKE, FAKE, k.get("lds", 128), 2, 100, 50, A, k.get("lda", 128), 1, k.get("n", 2),
                        k.get("d", d), W, b, 3, FAKE, k.get("ldy", 128), NULL]
    assert st(f, *args(lda=64)) == _lib.EINVAL                                   # ld_add < C
    assert st(f, *args(ldy=100)) == _lib.EINVAL                                  # ld_y < output width
    dw, Ww, bw = _mlp_args([128, 256, 64])
    assert st(f, *args(d=dw)) == _lib.EUNSUPPORTED                               # a layer wider than 128
    d6, W6, b6 = _mlp_args([6, 32])
    assert st(f, *args(d=d6, n=1, lds=8, lda=8, ldy=32)) == _lib.EUNSUPPORTED     # dims[0] % 4 != 0
    assert st(f, *args(lds=130)) == _lib.EUNSUPPORTED                            # ld_src % 4 != 0
    a = args()
    a[5] = 0
    assert st(f, *a) == _lib.OK                                                  # Nd = 0: nothing to do
    a = args()
    a[0] = NULL
    assert st(f, *a) == _lib.EINVAL                                              # NULL nit


def test_count_out_of_range_validation():
    f = "mesorasi_count_out_of_range"
    assert st(f, FAKE, -1, 10, FAKE, NULL) == _lib.EINVAL         # n < 0
    assert st(f, FAKE, 5, 10, NULL, NULL) == _lib.EINVAL          # NULL count
    assert st(f, NULL, 5, 10, FAKE, NULL) == _lib.EINVAL          # NULL idx with n > 0


def test_aggregate_mlp_validation():
    L = _lib.lib()
    f = "mesorasi_aggregate_mlp"
    d, W, b = _mlp_args([67, 64, 64, 128])
    args = lambda **k: [k.get("cxyz", FAKE), FAKE, k.get("ldp", 64), FAKE, FAKE, 2, 100, 10, k.get("K", 8),
                        k.get("C", 64), k.get("n", 3), k.get("d", d), W, b, 7, FAKE, k.get("ldy", 128), NULL, 0, NULL]
    assert st(f, *args(K=0)) == _lib.EINVAL                         # K < 1
    assert st(f, *args(C=60)) == _lib.EINVAL                        # dims[0] != 3 + C
    assert st(f, *args(ldp=32)) == _lib.EINVAL                      # ld_pft < C
    assert st(f, *args(cxyz=NULL)) == _lib.EINVAL                   # NULL cxyz
    dw, Ww, bw = _mlp_args([67, 64, 256])
    assert st(f, *args(d=dw, n=2, ldy=256)) == _lib.EUNSUPPORTED     # output wider than the fused kernel's
    assert b"narrow" in L.mesorasi_last_error()
    d1, _, _ = _mlp_args([67, 64])
    assert st(f, *args(d=d1, n=1)) == _lib.EUNSUPPORTED              # one layer
    d3, _, _ = _mlp_args([65, 64, 64])
    assert st(f, FAKE, FAKE, 62, FAKE, FAKE, 2, 100, 10, 8, 62, 2, d3, W, b, 7, FAKE, 128, NULL, 0, NULL) == \
        _lib.EUNSUPPORTED                                            # C not a multiple of 4

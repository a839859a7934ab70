"""ctypes loader for libmesorasi.so (the gfx950 HIP library).

Loading fails loudly when the library has not been built: there is no
fallback implementation of any entry point.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
# MESORASI_LIBRARY names another build of the same sources (the host
# sanitizer build of the test suite); unset, the in-tree library loads
LIB_PATH = os.environ.get("MESORASI_LIBRARY") or os.path.join(HERE, "libmesorasi.so")

OK, EINVAL, EUNSUPPORTED, EHIP, EWORKSPACE = 0, -1, -2, -3, -4
NOALLOC_WS_BYTES = 32 << 20    # MESORASI_NOALLOC_WS_BYTES: the allocation-free MLP's fixed scratch
F32, BF16 = 0, 1

_i64, _i32, _u32, _p, _f = ctypes.c_int64, ctypes.c_int32, ctypes.c_uint32, ctypes.c_void_p, ctypes.c_float
_size = ctypes.c_size_t

# name -> (restype, argtypes); mirrors include/mesorasi.h
SIGNATURES = {
    "mesorasi_version": (ctypes.c_int, []),
    "mesorasi_strerror": (ctypes.c_char_p, [ctypes.c_int]),
    "mesorasi_last_error": (ctypes.c_char_p, []),
    "mesorasi_fps": (ctypes.c_int, [_p, _i64, _i64, _i64, _p, _p, _p, _size, _p]),
    "mesorasi_fps_workspace": (_size, [_i64, _i64, _i64]),
    "mesorasi_fps_prefix": (ctypes.c_int, [_p, _p, _i64, _i64, _i64, _p, _p, _p]),
    "mesorasi_fps_prefix_levels": (ctypes.c_int, [_p, _p, _i64, _i64, ctypes.c_int32, _p, _p, _p, _p]),
    "mesorasi_ball_query": (ctypes.c_int, [_p, _p, _i64, _i64, _i64, _f, _i32, _p, _p, _p, _size, _p]),
    "mesorasi_ball_query_workspace": (_size, [_i64, _i64, _i64]),
    "mesorasi_ball_query_grid_workspace": (_size, [_i64, _i64]),
    "mesorasi_ball_query_grid_build": (ctypes.c_int, [_p, _i64, _i64, ctypes.c_float, _p, _size, _p]),
    "mesorasi_ball_query_grid": (ctypes.c_int, [_p, _p, _i64, _i64, _i64, ctypes.c_float, ctypes.c_int32, _p, _p, _p,
                                                _size, _p]),
    "mesorasi_knn": (ctypes.c_int, [_p, _i64, _p, _i64, _i64, _i64, _i64, _i32, _i32, _p, _p, _p]),
    "mesorasi_pointwise_mlp": (ctypes.c_int, [_p, _i32, _i64, _p, _i32, _i64, _i64, _i32, _p, _p, _p, _u32, _i32,
                                              _i32, _p, _i64, _i64, _p, _size, _p]),
    "mesorasi_pointwise_mlp_workspace": (_size, [_i64, _i32, _p, _i32, _i64]),
    "mesorasi_pointwise_mlp_noalloc": (ctypes.c_int, [_p, _i32, _i64, _p, _i32, _i64, _i64, _i32, _p, _p, _p, _u32,
                                                      _i32, _i32, _p, _i64, _i64, _p]),
    "mesorasi_aggregate_max": (ctypes.c_int, [_p, _i64, _i32, _p, _i64, _i64, _i64, _i32, _i32, _p, _p, _i64, _i32,
                                              _i32, _p, _i64, _p]),
    "mesorasi_conventional_module": (ctypes.c_int, [_p, _p, _i32, _i64, _p, _p, _i64, _i64, _i64, _i32, _i32, _i32,
                                                    _p, _p, _p, _u32, _i32, _p, _i64, _p, _size, _p]),
    "mesorasi_conventional_workspace": (_size, [_i64, _i64, _i32, _i32, _p, _i32]),
    "mesorasi_ltd_module": (ctypes.c_int, [_p, _i64, _p, _i64, _p, _p, _i64, _i64, _i64, _i32, _i32, _i32, _p, _p, _p,
                                           ctypes.c_uint32, _i32, _p, _i64, _p, _size, _p]),
    "mesorasi_ltd_workspace": (_size, [_i64, _i64, _i32, _i32, _p, _i32]),
    "mesorasi_interpolate3": (ctypes.c_int, [_p, _p, _p, _i64, _i64, _i64, _i64, _i32, _p, _i64, _p]),
    "mesorasi_three_nn": (ctypes.c_int, [_p, _p, _i64, _i64, _i64, _p, _p, _p]),
    "mesorasi_interpolate3_apply": (ctypes.c_int, [_p, _p, _p, _i64, _i64, _i64, _i64, _i32, _p, _i64, _p]),
    "mesorasi_interpolate3_add": (ctypes.c_int, [_p, _p, _p, _i64, _i64, _i64, _i64, _i32, _p, _i64, _i32, _p, _i64,
                                                 _p]),
    "mesorasi_interpolate3_mlp": (ctypes.c_int, [_p, _p, _p, _i64, _i64, _i64, _i64, _p, _i64, _i32, _i32, _p, _p, _p,
                                                 _u32, _p, _i64, _p]),
    "mesorasi_cast_bf16": (ctypes.c_int, [_p, _i64, _p, _p]),
    "mesorasi_edgeconv_fold": (ctypes.c_int, [_p, _p, _i32, _i32, _p, _p, _p]),
    "mesorasi_count_out_of_range": (ctypes.c_int, [_p, _i64, _i32, _p, _p]),
    "mesorasi_aggregate_mlp": (ctypes.c_int, [_p, _p, _i64, _p, _p, _i64, _i64, _i64, _i32, _i32, _i32, _p, _p, _p,
                                              _u32, _p, _i64, _p, _i64, _p]),
}

_lib = None


def lib():
    """The loaded library; raises if libmesorasi.so is missing."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build() (or "
                               f"python paper_2008_06967_amd/build.py) first")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


class MesorasiError(RuntimeError):
    def __init__(self, status: int, where: str):
        L = lib()
        self.status = status
        msg = L.mesorasi_strerror(status).decode()
        detail = L.mesorasi_last_error().decode()
        super().__init__(f"{where}: {msg} ({status}): {detail}")


def check(status: int, where: str) -> None:
    if status != OK:
        raise MesorasiError(status, where)

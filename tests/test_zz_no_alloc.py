"""The allocation-free MLP entry point (mesorasi_pointwise_mlp_noalloc,
scratch in a fixed per-GPU device array) against mesorasi_pointwise_mlp
with a caller workspace: the same kernels run, so the outputs must be
identical, and they meet the oracle's tolerance.  Each case makes two
calls in a row on the shared array, the second with a smaller input, so
stale contents of the first call would show in the second."""
import ctypes

import numpy as np
import pytest
import torch

import oracle as O
from paper_2008_06967_amd import _lib, ops
from paper_2008_06967_amd._lib import BF16, F32

pytestmark = pytest.mark.gpu

TOL = {F32: 1e-4, BF16: 2e-2}


def _rng(s):
    return np.random.default_rng(np.random.SeedSequence([200806967, 77, s]))


def _params(r, dims, dt):
    Ws = [(r.standard_normal((dims[l + 1], dims[l])) * np.sqrt(2.0 / dims[l])).astype(np.float32)
          for l in range(len(dims) - 1)]
    bs = [r.uniform(-0.1, 0.1, dims[l + 1]).astype(np.float32) for l in range(len(dims) - 1)]
    return Ws, bs, ops.MLPParams(Ws, bs, dt)


def _normwise(g, r):
    g, r = np.asarray(g, np.float64), np.asarray(r, np.float64)
    return float(np.max(np.abs(g - r)) / max(np.max(np.abs(r)), 1e-30))


def _host(t):
    return (t.float() if t.dtype == torch.bfloat16 else t).cpu().numpy()


# (name, dims, dtype, pool_group, first rows, second rows, x0 width or 0 for one source)
CASES = [
    ("sa2_f32", [131, 128, 128, 256], F32, 0, 16384, 3000, 3),      # 16 MiB of activations
    ("split_k_f32", [67, 200, 64], F32, 0, 2000, 700, 0),           # small row counts: split-K partials
    ("bf16", [64, 128, 128, 256], BF16, 0, 8192, 300, 0),
    ("pooled_group_all", [259, 256, 512, 1024], F32, 128, 4096, 1024, 3),
]


@pytest.mark.parametrize("name,dims,dt,G,rows1,rows2,c0", CASES, ids=[c[0] for c in CASES])
def test_noalloc_matches_workspace_entry_point(gpu, name, dims, dt, G, rows1, rows2, c0):
    r = _rng(len(name))
    Ws, bs, p = _params(r, dims, dt)
    need = ops.mlp_workspace_bytes(rows1, p, G)
    assert 0 < need <= _lib.NOALLOC_WS_BYTES
    for rows in (rows1, rows2):
        x = r.standard_normal((rows, dims[0])).astype(np.float32)
        tx = torch.from_numpy(x).cuda()
        if c0:
            a, b = tx[:, :c0].contiguous(), tx[:, c0:].contiguous()
            ref = ops.pointwise_mlp(a, p, b, pool_group=G)
            torch.cuda.synchronize()
            got = ops.pointwise_mlp_noalloc(a, p, b, pool_group=G)
        else:
            ref = ops.pointwise_mlp(tx, p, pool_group=G)
            torch.cuda.synchronize()
            got = ops.pointwise_mlp_noalloc(tx, p, pool_group=G)
        torch.cuda.synchronize()
        assert torch.equal(got, ref), f"{name}: rows {rows}"
        if rows == rows2:
            o = O.mlp(x, Ws, bs, bf16=dt == BF16)
            if G:
                o = O.rowgroup_max(o.reshape(1, rows, -1), G)[0]
            assert _normwise(_host(got), o) <= TOL[dt], f"{name}: rows {rows}"


def test_noalloc_rejects_more_than_its_scratch(gpu):
    """A call that would need more than the fixed array is refused before
    anything is launched; the output keeps its contents."""
    dims = [131, 128, 128, 256]
    r = _rng(5)
    _, _, p = _params(r, dims, F32)
    rows = 40000
    assert ops.mlp_workspace_bytes(rows, p) > _lib.NOALLOC_WS_BYTES
    x = torch.zeros((rows, 131), device="cuda")
    y = torch.full((rows, 256), 7.0, device="cuda")
    d, W, b = p.abi()
    rc = _lib.lib().mesorasi_pointwise_mlp_noalloc(x.data_ptr(), 131, 131, None, 0, 0, rows, 3, d, W, b, 7, F32, F32,
                                                    y.data_ptr(), 256, 0, ctypes.c_void_p(0))
    assert rc == _lib.EUNSUPPORTED
    assert b"scratch" in _lib.lib().mesorasi_last_error()
    torch.cuda.synchronize()
    assert bool((y == 7.0).all())

"""Host-side logic of bench.py (no GPU): the algorithmic work each call is
credited with, and the staleness rule of the recorded HBM traffic."""
import hashlib
import os
import sys
import types

import numpy as np
import pytest
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_fps_work_and_latency_fields():
    xyz = torch.zeros(3, 100, 3)
    kind, amount, extra = bench.call_work("fps", (xyz, 10), {})
    assert kind == "alu"
    assert amount == pytest.approx(8.0 * 3 * 9 * 100 / 1e12)
    assert extra == {"serial_iterations": 9, "workgroups": 3}


def test_ball_query_work_counts_the_scanned_pairs():
    """A query whose K slots fill scans up to its K-th hit; a short list
    (padded with its first hit) scans all N points.  Without the output
    the worst case B * M * N is credited."""
    xyz, q = torch.zeros(2, 50, 3), torch.zeros(2, 3, 3)
    K = 4
    nit = torch.tensor([[[0, 3, 9, 12], [5, 5, 5, 5], [1, 2, 3, 4]],
                        [[7, 7, 7, 7], [10, 20, 30, 49], [0, 1, 2, 3]]], dtype=torch.int32)
    kind, amount, extra = bench.call_work("ball_query", (xyz, q, 0.1, K), {}, (nit, None))
    scanned = 13 + 50 + 5 + 50 + 50 + 4
    assert kind == "alu"
    assert extra["scanned_pairs"] == scanned
    assert amount == pytest.approx(8.0 * scanned / 1e12)
    assert extra["worst_case_pairs"] == 2 * 3 * 50
    assert extra["compulsory_bytes"] == 12 * 2 * 50 + 12 * 2 * 3 + 4 * 2 * 3 * K
    _, amount, _ = bench.call_work("ball_query", (xyz, q, 0.1, K), {})
    assert amount == pytest.approx(8.0 * 2 * 3 * 50 / 1e12)


def test_knn_self_query_reads_the_reference_once():
    ref = torch.zeros(2, 40, 8)
    _, amount, extra = bench.call_work("knn", (ref, ref, 5), {})
    assert amount == pytest.approx(3.0 * 8 * 2 * 40 * 40 / 1e12)
    assert extra["compulsory_bytes"] == 4 * 2 * 40 * 8 + 4 * 2 * 40 * 5
    q = torch.zeros(2, 10, 8)
    _, _, extra = bench.call_work("knn", (ref, q, 5), {})
    assert extra["compulsory_bytes"] == 4 * 2 * 40 * 8 + 4 * 2 * 10 * 8 + 4 * 2 * 10 * 5


def test_mlp_work_sums_every_layer():
    prm = types.SimpleNamespace(dims=[3, 64, 64, 128], dtype=0)
    x0 = torch.zeros(4, 256, 3)
    out = torch.zeros(4, 256, 128)
    kind, amount, extra = bench.call_work("pointwise_mlp", (x0, prm), {}, out)
    assert kind == "mfma"
    assert amount == pytest.approx(2.0 * 1024 * (3 * 64 + 64 * 64 + 64 * 128) / 1e12)
    # compulsory bytes of a fused MLP: input rows, output rows, weights
    assert extra["compulsory_bytes_mlp"] == 1024 * 3 * 4 + 1024 * 128 * 4 + (3 * 64 + 64 * 64 + 64 * 128) * 4
    assert extra["bf16"] is False


def test_aggregation_compulsory_bytes():
    pft = torch.zeros(2, 30, 16)
    nit = torch.zeros(2, 5, 4, dtype=torch.int32)
    cidx = torch.zeros(2, 5, dtype=torch.int32)
    kind, amount, extra = bench.call_work("aggregate_max", (pft, nit, cidx, None), {})
    assert kind == "hbm"
    assert amount * 1e9 == pytest.approx(2 * 30 * 16 * 4 + 4 * 2 * 5 * 4 + 4 * 2 * 5 * 16 + 4 * 2 * 5)
    assert extra["logical_gather_bytes"] == 2 * 5 * 4 * 16 * 4


def test_recorded_traffic_matches_its_source_hash():
    """Every entry either names the current hash of its kernel source (and
    is returned as fetch + write) or is reported as absent."""
    path = os.path.join(ROOT, "profiles", "pmc_traffic.txt")
    for line in open(path):
        if line.startswith("#") or not line.strip():
            continue
        key, fetch, write, h, src = line.split()[:5]
        cur = hashlib.sha256(open(os.path.join(ROOT, "paper_2008_06967_amd", "csrc", src), "rb").read()).hexdigest()[:16]
        got = bench.load_traffic(key)
        if cur == h:
            assert got == {"fetch_bytes": float(fetch), "write_bytes": float(write),
                           "bytes": float(fetch) + float(write)}
        else:
            assert got is None
    assert bench.load_traffic("no_such_kernel#0@nowhere") is None


def test_cpu_threads_respects_the_job_share(monkeypatch):
    avail = len(os.sched_getaffinity(0))
    monkeypatch.setenv("OMP_NUM_THREADS", "1")
    assert bench.cpu_threads() == (1, avail)
    monkeypatch.delenv("OMP_NUM_THREADS")
    assert bench.cpu_threads() == (avail, avail)


def test_interpolation_bytes():
    """Source rows once, 3 neighbours and distances per destination, the
    output; the add form also reads the added rows."""
    nit = torch.zeros(2, 100, 3, dtype=torch.int32)
    f = torch.zeros(2, 25, 16)
    kind, amount, extra = bench.call_work("interpolate3_apply", (nit, None, f), {})
    base = 4 * 2 * 25 * 16 + 24 * 2 * 100 + 4 * 2 * 100 * 16
    assert kind == "hbm" and amount == pytest.approx(base / 1e9)
    assert extra["logical_gather_bytes"] == 12 * 2 * 100 * 16
    kind, amount, _ = bench.call_work("interpolate3_add", (nit, None, f, torch.zeros(2, 100, 16)), {})
    assert kind == "hbm" and amount == pytest.approx((base + 4 * 2 * 100 * 16) / 1e9)


def test_interpolate3_mlp_work_is_the_mlp():
    prm = types.SimpleNamespace(dims=[128, 128, 128], dtype=0)
    nit = torch.zeros(2, 1000, 3, dtype=torch.int32)
    kind, amount, _ = bench.call_work("interpolate3_mlp", (nit, None, None, None, prm), {})
    assert kind == "mfma" and amount == pytest.approx(2.0 * 2000 * (128 * 128 * 2) / 1e12)

"""CPU model of the multi-workgroup FPS exchange (threads stand in for the
workgroups of one cloud), checked against the oracle.

Protocol (one cloud, G workgroups, workgroup g owns the contiguous points
[g*S, (g+1)*S)):
  * the slot table holds 2 x G slots and is cleared before the launch;
  * iteration m >= 1: every workgroup updates its running minima with the
    newest centroid, finds its local winner (largest minimum, lowest index
    on ties), and publishes it in slot [m % 2][g]: four words, each tagged
    with m, carrying (distance, index), x, y and z;
  * it then waits until all G slots [m % 2][*] carry tag m, and takes the
    winner: the largest distance, the lowest g on ties (g orders indices,
    so that is the lowest index);
  * a workgroup can only publish iteration m + 2 (reusing parity m % 2)
    after it has seen every slot of iteration m + 1, which each workgroup
    writes only after it has read every slot of iteration m: two parities
    suffice, and a tag never matches stale contents.
The model interleaves the threads with random delays and checks every read
against the invariants above."""
import random
import threading

import numpy as np
import pytest

import oracle as O


def _dist(a, b):
    # the fp32 chain of the distance reading: t = a - b, d = fma(t, t, d)
    d = np.float32(0.0)
    for c in range(3):
        t = np.float32(a[c] - b[c])
        d = np.float32(np.float64(t) * np.float64(t) + np.float64(d))
    return d


def _multi_wg_fps(xyz, M, G, seed):
    N = xyz.shape[0]
    S = -(-N // G)
    slots = [[None] * G for _ in range(2)]       # (tag, dist, index, x, y, z)
    lock = threading.Lock()
    out = [None] * M
    errors = []
    rnd = random.Random(seed)

    def wg(g):
        lo, hi = g * S, min(N, (g + 1) * S)
        dmin = [np.float32(np.inf)] * (hi - lo)
        c = xyz[0]
        if g == 0:
            out[0] = 0
        for m in range(1, M):
            best_d, best_j = np.float32(-1.0), -1
            for q in range(hi - lo):
                d = _dist(xyz[lo + q], c)
                if d < dmin[q]:
                    dmin[q] = d
                if dmin[q] > best_d:                # strict: the lowest index keeps a tie
                    best_d, best_j = dmin[q], lo + q
            if rnd.random() < 0.3:
                threading.Event().wait(rnd.random() * 1e-3)
            px = xyz[best_j] if best_j >= 0 else np.zeros(3, np.float32)
            with lock:
                slots[m % 2][g] = (m, best_d, best_j, px[0], px[1], px[2])
            while True:
                with lock:
                    seen = list(slots[m % 2])
                if all(s is not None and s[0] == m for s in seen):
                    break
                for s in seen:
                    # a slot holds iteration m - 2 (not yet overwritten) or m:
                    # never a later one, which would mean a lost value
                    if s is not None and s[0] not in (m, m - 2):
                        errors.append((g, m, s[0]))
                threading.Event().wait(1e-5)
            w = max(range(G), key=lambda h: (seen[h][1], -h))   # largest distance, lowest g
            _, _, j, x, y, z = seen[w]
            c = np.array([x, y, z], np.float32)
            if g == 0:
                out[m] = j

    ts = [threading.Thread(target=wg, args=(g,)) for g in range(G)]
    for t in ts:
        t.start()
    for t in ts:
        t.join()
    assert not errors, errors[:5]
    return np.array(out, np.int32)


@pytest.mark.parametrize("G,N,M,kind", [(4, 64, 20, "uniform"), (8, 61, 30, "grid"), (3, 40, 40, "dups")])
def test_multi_workgroup_protocol_matches_oracle(G, N, M, kind):
    r = np.random.default_rng(G * 100 + N)
    if kind == "grid":
        xyz = r.integers(0, 3, (N, 3)).astype(np.float32)      # many equal distances
    elif kind == "dups":
        base = r.uniform(-1, 1, (N // 4, 3))
        xyz = base[r.integers(0, N // 4, N)].astype(np.float32)  # duplicates: dmin reaches 0
    else:
        xyz = r.uniform(-1, 1, (N, 3)).astype(np.float32)
    ref, _ = O.fps(xyz[None], M)
    got = _multi_wg_fps(xyz, M, G, seed=N)
    assert np.array_equal(got, ref[0])

"""CPU checks of the test-side kNN near-tie check: it accepts mismatches
that rounding of the search input explains and rejects a planted
selection error."""
import numpy as np
import pytest

import oracle as O
from knn_checks import check_knn_near_ties


def _layers(seed, noise):
    """Two 'layers': layer 0 (exact, same input), layer 1 searched on a
    perturbed copy of layer 0's output (the GPU side) and on the output
    itself (the oracle side).  Pairs of near-duplicate points make ties
    that the perturbation flips."""
    r = np.random.default_rng(seed)
    base = r.standard_normal((1, 150, 16))
    X = np.concatenate([base, base + 1e-6 * r.standard_normal(base.shape)], 1).astype(np.float32)
    Xg = (X + noise * r.standard_normal(X.shape)).astype(np.float32)
    K = 10
    n0, _ = O.knn(X, X, K)
    ref = {"layers": [{"nit": n0, "out": X}, {"nit": O.knn(X, X, K)[0], "out": X}]}
    got = {"nit0": n0.copy(), "x0": Xg, "nit1": O.knn(Xg, Xg, K)[0]}
    return got, ref, K


def test_near_ties_accepted():
    got, ref, K = _layers(1, 3e-7)
    counts = check_knn_near_ties(got, ref, K, "cpu", max_frac=1.0)
    assert counts[1] > 0          # the perturbation did flip some near-ties


def test_planted_selection_error_rejected():
    got, ref, K = _layers(1, 3e-7)
    nit = got["nit1"]
    q, s = 7, K - 1
    far = np.argmax(np.linalg.norm(ref["layers"][0]["out"][0] - ref["layers"][0]["out"][0, q], axis=-1))
    nit[0, q, s] = far
    with pytest.raises(AssertionError):
        check_knn_near_ties(got, ref, K, "cpu", max_frac=1.0)


def test_layer0_mismatch_rejected():
    got, ref, K = _layers(2, 0.0)
    got["nit0"][0, 3, 2] = got["nit0"][0, 3, 1]
    with pytest.raises(AssertionError):
        check_knn_near_ties(got, ref, K, "cpu", max_frac=1.0)

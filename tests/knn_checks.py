"""Shared check for kNN results computed on inputs that differ from the
oracle's by rounding (DGCNN free running): every differing entry must be a
near-tie that the input difference explains."""
import numpy as np


def check_knn_near_ties(got, ref, K, label, max_frac=0.001):
    """Free-running DGCNN: layer l >= 1 searches the GPU's layer l - 1
    output, which differs from the oracle's by rounding, so a few kNN
    entries may differ.  Each differing (query, slot) must be explained by
    that input difference: with D the exact Euclidean distance on the
    oracle's input, eta = 2 sqrt(C) max|X_gpu - X_oracle| bounds how far
    any distance moves between the two inputs, and the s-th smallest of
    two sets of distances within eps of each other differ by at most eps,
    so |D(q, j_gpu) - D(q, j_oracle)| <= 2 eta + 4 rho (rho: the fp32
    chain's rounding, (C + 2) 2^-24 of the K-th distance).  At most
    max_frac of a layer's entries may differ.  Returns the mismatch counts
    per layer."""
    counts = []
    u = 2.0 ** -24
    for l, r in enumerate(ref["layers"]):
        bad = np.argwhere(got[f"nit{l}"] != r["nit"])
        counts.append(len(bad))
        if l == 0:
            assert len(bad) == 0, f"{label}: layer 0 searches xyz and must be exact"
            continue
        assert len(bad) <= max_frac * r["nit"].size, f"{label} layer {l}: {len(bad)} kNN entries differ"
        if len(bad) == 0:
            continue
        X = ref["layers"][l - 1]["out"].astype(np.float64)
        Xg = got[f"x{l - 1}"].astype(np.float64)
        C = X.shape[-1]
        eta = 2.0 * np.sqrt(C) * float(np.max(np.abs(Xg - X)))
        gaps = []
        for b, q, s in bad:
            jg, jr, jk = got[f"nit{l}"][b, q, s], r["nit"][b, q, s], r["nit"][b, q, K - 1]
            dg = np.linalg.norm(X[b, q] - X[b, jg])
            dr = np.linalg.norm(X[b, q] - X[b, jr])
            dk = np.linalg.norm(X[b, q] - X[b, jk])
            rho = (C + 2) * u * (dk + eta)
            assert abs(dg - dr) <= 2 * eta + 4 * rho + 1e-30, \
                f"{label} layer {l} cloud {b} query {q} slot {s}: |{dg} - {dr}| > 2 * {eta} + 4 * {rho}"
            gaps.append(abs(dg - dr) / max(dk, 1e-30))
        print(f"{label} layer {l}: {len(bad)} of {r['nit'].size} kNN entries differ, all near-ties "
              f"(max relative distance gap {max(gaps):.2e}, eta {eta:.2e})", flush=True)
    return counts

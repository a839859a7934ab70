/*
 * CPU oracle for delayed-aggregation point-cloud modules -- TEST
 * INFRASTRUCTURE ONLY (see oracle.h).  Plain scalar C, single thread,
 * built with -O2 -ffp-contract=off -fno-fast-math so that every float
 * operation below is one IEEE-754 binary32 (or binary64) operation in the
 * order written.
 *
 * Paper sections followed (Feng et al., arXiv 2008.06967):
 *  - module N -> A -> F -> reduce: Sec. 3.1 "Module Internals", Eq. (1)
 *  - delayed-aggregation, PFT and NIT: Sec. 4.1, Eq. (2)-(3), walk-through
 *  - max/subtract distributivity: Sec. 4.1, last paragraph of walk-through
 *  - aggregation loop over NIT entries: Sec. 5.2, first paragraph
 *  - sampling / grouping / three_interpolate kernels of the PointNet++
 *    baselines: Sec. 6, "Software Setup"
 */
#include "oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

/* Squared distance with a fixed operation order (reading of the paper's
 * unspecified distance metric; see the header). */
float orc_dist2(const float* a, const float* b, int C) {
    float d = 0.0f;
    for (int c = 0; c < C; ++c) {
        float t = a[c] - b[c];
        d = fmaf(t, t, d);
    }
    return d;
}

/* fp32 -> bf16 with round-to-nearest-even, returned widened back to fp32.
 * Inputs are finite (the oracle never feeds NaN/Inf). */
float orc_bf16_round(float f) {
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    uint32_t lsb = (u >> 16) & 1u;
    u = (u + 0x7fffu + lsb) & 0xffff0000u;
    memcpy(&f, &u, sizeof f);
    return f;
}

/* ------------------------------------------------------------------------
 * Farthest-point sampling.  The paper names the sampling step of its
 * PointNet++ baselines (Sec. 6, Software Setup) without defining it; this is
 * the standard greedy definition: keep, for every point, its distance to the
 * nearest already-selected point, and select the point where that distance
 * is largest.  Start at index 0, lowest index wins a tie.
 * ---------------------------------------------------------------------- */
void orc_fps(const float* xyz, int64_t B, int64_t N, int64_t M, int32_t* idx, float* cxyz) {
    float* dmin = (float*)malloc(sizeof(float) * (size_t)N);
    for (int64_t b = 0; b < B; ++b) {
        const float* p = xyz + b * N * 3;
        for (int64_t j = 0; j < N; ++j) dmin[j] = INFINITY;
        int64_t sel = 0;
        idx[b * M] = 0;
        for (int64_t m = 1; m < M; ++m) {
            const float* c = p + sel * 3;
            int64_t best = 0;
            float bestd = -1.0f;
            for (int64_t j = 0; j < N; ++j) {
                float d = orc_dist2(p + j * 3, c, 3);
                if (d < dmin[j]) dmin[j] = d;
                if (dmin[j] > bestd) {
                    bestd = dmin[j];
                    best = j;
                }
            }
            sel = best;
            idx[b * M + m] = (int32_t)sel;
        }
        if (cxyz) {
            for (int64_t m = 0; m < M; ++m)
                for (int c = 0; c < 3; ++c) cxyz[(b * M + m) * 3 + c] = p[(int64_t)idx[b * M + m] * 3 + c];
        }
    }
    free(dmin);
}

/* The same selection rule recomputed from scratch at every step:
 * sel[m] = argmax_j min_{i<m} dist2(x_j, x_sel[i]).  O(M^2 N); used only to
 * pin orc_fps on small inputs. */
void orc_fps_bruteforce(const float* xyz, int64_t B, int64_t N, int64_t M, int32_t* idx) {
    for (int64_t b = 0; b < B; ++b) {
        const float* p = xyz + b * N * 3;
        idx[b * M] = 0;
        for (int64_t m = 1; m < M; ++m) {
            int64_t best = 0;
            float bestd = -1.0f;
            for (int64_t j = 0; j < N; ++j) {
                float mn = INFINITY;
                for (int64_t i = 0; i < m; ++i) {
                    float d = orc_dist2(p + j * 3, p + (int64_t)idx[b * M + i] * 3, 3);
                    if (d < mn) mn = d;
                }
                if (mn > bestd) {
                    bestd = mn;
                    best = j;
                }
            }
            idx[b * M + m] = (int32_t)best;
        }
    }
}

/* ------------------------------------------------------------------------
 * Ball query (neighbor search N of Eq. (1); Sec. 3.1 "Neighbor Search").
 * First K points in index order strictly inside the radius; remaining slots
 * repeat the first hit.  cnt = number of real hits (<= K); scanned = number
 * of candidates examined before the K-th hit (N when fewer than K hits).
 * ---------------------------------------------------------------------- */
void orc_ball_query(const float* xyz, const float* qxyz, int64_t B, int64_t N, int64_t M, float radius,
                    int32_t K, int32_t* nit, int32_t* cnt, int64_t* scanned) {
    const float r2 = radius * radius;
    for (int64_t b = 0; b < B; ++b) {
        const float* p = xyz + b * N * 3;
        for (int64_t m = 0; m < M; ++m) {
            const float* q = qxyz + (b * M + m) * 3;
            int32_t* row = nit + (b * M + m) * K;
            int32_t n = 0;
            int64_t j = 0;
            for (; j < N && n < K; ++j) {
                if (orc_dist2(p + j * 3, q, 3) < r2) row[n++] = (int32_t)j;
            }
            int32_t pad = n > 0 ? row[0] : 0;
            for (int32_t k = n; k < K; ++k) row[k] = pad;
            if (cnt) cnt[b * M + m] = n;
            if (scanned) scanned[b * M + m] = j;
        }
    }
}

/* ------------------------------------------------------------------------
 * k nearest neighbours in C-dimensional space (DGCNN search in the previous
 * module's output space, Sec. 5.1 "Work Flow"; PointNet++ 3-NN
 * interpolation).  Output sorted by (dist2, index); self included.
 * Insertion into a sorted list of K; candidates arrive in ascending index
 * order, so a strict '<' keeps equal distances in index order.
 * ---------------------------------------------------------------------- */
void orc_knn(const float* ref, int64_t ld_ref, const float* query, int64_t ld_query, int64_t B, int64_t N,
             int64_t M, int32_t C, int32_t K, int32_t* nit, float* dist) {
    float* bd = (float*)malloc(sizeof(float) * (size_t)K);
    int32_t* bj = (int32_t*)malloc(sizeof(int32_t) * (size_t)K);
    for (int64_t b = 0; b < B; ++b) {
        for (int64_t m = 0; m < M; ++m) {
            const float* q = query + (b * M + m) * ld_query;
            int32_t have = 0;
            for (int64_t j = 0; j < N; ++j) {
                float d = orc_dist2(ref + (b * N + j) * ld_ref, q, C);
                if (have == K && !(d < bd[K - 1])) continue;
                int32_t pos = have < K ? have : K - 1;
                while (pos > 0 && d < bd[pos - 1]) {
                    bd[pos] = bd[pos - 1];
                    bj[pos] = bj[pos - 1];
                    --pos;
                }
                bd[pos] = d;
                bj[pos] = (int32_t)j;
                if (have < K) ++have;
            }
            for (int32_t k = 0; k < K; ++k) {
                nit[(b * M + m) * K + k] = bj[k];
                if (dist) dist[(b * M + m) * K + k] = bd[k];
            }
        }
    }
    free(bd);
    free(bj);
}

/* ------------------------------------------------------------------------
 * Shared per-point MLP (feature computation F, Sec. 3.1 "Feature
 * Computation"; Eq. (3) with phi = ReLU).  y is [rows, dims[n_layers]].
 * ---------------------------------------------------------------------- */
void orc_mlp(const float* x, int64_t rows, int32_t n_layers, const int32_t* dims, const float* const* W,
             const float* const* bias, uint32_t relu_mask, int32_t bf16, float* y) {
    int32_t wmax = 0;
    for (int32_t l = 0; l <= n_layers; ++l)
        if (dims[l] > wmax) wmax = dims[l];
    float* Wr[32];
    for (int32_t l = 0; l < n_layers; ++l) {
        size_t n = (size_t)dims[l] * (size_t)dims[l + 1];
        Wr[l] = (float*)malloc(sizeof(float) * n);
        for (size_t i = 0; i < n; ++i) Wr[l][i] = bf16 ? orc_bf16_round(W[l][i]) : W[l][i];
    }
    float* a = (float*)malloc(sizeof(float) * (size_t)wmax);
    float* h = (float*)malloc(sizeof(float) * (size_t)wmax);
    for (int64_t r = 0; r < rows; ++r) {
        for (int32_t i = 0; i < dims[0]; ++i) {
            float v = x[r * dims[0] + i];
            a[i] = bf16 ? orc_bf16_round(v) : v;
        }
        for (int32_t l = 0; l < n_layers; ++l) {
            const int32_t cin = dims[l], cout = dims[l + 1];
            for (int32_t o = 0; o < cout; ++o) {
                double acc = 0.0;
                const float* w = Wr[l] + (size_t)o * (size_t)cin;
                for (int32_t i = 0; i < cin; ++i) acc += (double)a[i] * (double)w[i];
                if (bias && bias[l]) acc += (double)bias[l][o];
                float v = (float)acc;
                if (relu_mask & (1u << l)) v = v > 0.0f ? v : 0.0f;
                h[o] = bf16 ? orc_bf16_round(v) : v;
            }
            float* t = a;
            a = h;
            h = t;
        }
        memcpy(y + r * dims[n_layers], a, sizeof(float) * (size_t)dims[n_layers]);
    }
    free(a);
    free(h);
    for (int32_t l = 0; l < n_layers; ++l) free(Wr[l]);
}

/* ------------------------------------------------------------------------
 * Aggregation A on the point feature table (Sec. 5.2 first paragraph;
 * Sec. 4.1 max/subtract distributivity): for each NIT entry gather the K
 * PFT rows, reduce them column-wise with max, then combine with the
 * centroid's row: out = max + sign * centroid (sign -1 for PointNet++
 * offsets, +1 for the DGCNN x_i term).  Centroid row from cidx (a PFT row),
 * from an explicit table cfeat [B*M, ld_c], or absent when both are NULL.
 * ---------------------------------------------------------------------- */
void orc_aggregate_max(const float* pft, int64_t ld_pft, const int32_t* nit, int64_t B, int64_t N, int64_t M,
                       int32_t K, int32_t C, const int32_t* cidx, const float* cfeat, int64_t ld_c,
                       int32_t sign, int32_t relu, float* out, int64_t ld_out) {
    for (int64_t b = 0; b < B; ++b) {
        for (int64_t m = 0; m < M; ++m) {
            const int32_t* row = nit + (b * M + m) * K;
            for (int32_t ch = 0; ch < C; ++ch) {
                float mx = pft[(b * N + row[0]) * ld_pft + ch];
                for (int32_t k = 1; k < K; ++k) {
                    float v = pft[(b * N + row[k]) * ld_pft + ch];
                    if (v > mx) mx = v;
                }
                float r = mx;
                if (cidx || cfeat) {
                    float cen = cidx ? pft[(b * N + cidx[b * M + m]) * ld_pft + ch] : cfeat[(b * M + m) * ld_c + ch];
                    r = sign < 0 ? mx - cen : mx + cen;
                }
                if (relu) r = r > 0.0f ? r : 0.0f;
                out[(b * M + m) * ld_out + ch] = r;
            }
        }
    }
}

/* ------------------------------------------------------------------------
 * Conventional aggregation before F (Eq. (1); Sec. 3.1 "Aggregation"):
 * build the neighbor feature matrix, one row per (centroid, neighbor).
 *  - pointnet: [x_j - c, f_j]            (dims[0] = 3 + cf)
 *  - offsets : [x_j - x_c, f_j - f_c]    (whole-vector offsets p_k - p_i,
 *              centroid c = point cidx)
 *  - edge    : [f_i, f_j - f_i]          (DGCNN edge features, M = N)
 * ---------------------------------------------------------------------- */
void orc_group_pointnet(const float* xyz, const float* feat, int32_t cf, int64_t ld_f, const float* cxyz,
                        const int32_t* nit, int64_t B, int64_t N, int64_t M, int32_t K, float* nfm) {
    const int64_t cin = 3 + cf;
    for (int64_t b = 0; b < B; ++b)
        for (int64_t m = 0; m < M; ++m)
            for (int32_t k = 0; k < K; ++k) {
                const int64_t j = nit[(b * M + m) * K + k];
                float* o = nfm + ((b * M + m) * K + k) * cin;
                for (int c = 0; c < 3; ++c) o[c] = xyz[(b * N + j) * 3 + c] - cxyz[(b * M + m) * 3 + c];
                for (int32_t c = 0; c < cf; ++c) o[3 + c] = feat[(b * N + j) * ld_f + c];
            }
}

void orc_group_offsets(const float* xyz, const float* feat, int32_t cf, int64_t ld_f, const int32_t* cidx,
                       const int32_t* nit, int64_t B, int64_t N, int64_t M, int32_t K, float* nfm) {
    const int64_t cin = 3 + cf;
    for (int64_t b = 0; b < B; ++b)
        for (int64_t m = 0; m < M; ++m) {
            const int64_t ci = cidx[b * M + m];
            for (int32_t k = 0; k < K; ++k) {
                const int64_t j = nit[(b * M + m) * K + k];
                float* o = nfm + ((b * M + m) * K + k) * cin;
                for (int c = 0; c < 3; ++c) o[c] = xyz[(b * N + j) * 3 + c] - xyz[(b * N + ci) * 3 + c];
                for (int32_t c = 0; c < cf; ++c)
                    o[3 + c] = feat[(b * N + j) * ld_f + c] - feat[(b * N + ci) * ld_f + c];
            }
        }
}

void orc_group_edge(const float* f, int64_t ld_f, int32_t C, const int32_t* nit, int64_t B, int64_t N,
                    int32_t K, float* nfm) {
    for (int64_t b = 0; b < B; ++b)
        for (int64_t i = 0; i < N; ++i)
            for (int32_t k = 0; k < K; ++k) {
                const int64_t j = nit[(b * N + i) * K + k];
                float* o = nfm + ((b * N + i) * K + k) * (2 * (int64_t)C);
                const float* fi = f + (b * N + i) * ld_f;
                const float* fj = f + (b * N + j) * ld_f;
                for (int32_t c = 0; c < C; ++c) {
                    o[c] = fi[c];
                    o[C + c] = fj[c] - fi[c];
                }
            }
}

/*
 * Limited delayed aggregation (Sec. 7.3, "Ltd"): only the first layer's
 * matrix product is hoisted before aggregation, which keeps the module
 * exact because that product is linear.  With the PointNet++ grouping row
 * [x_j - x_c | f_j], the first layer's pre-activation is
 *   W1 [x_j | f_j] - W1[:, :3] x_c + b1 = P1[j] - Q[c] + b1,
 * where P1 = [x | f] W1^T is computed once per input point and Q[c] is the
 * centroid's term.  This routine forms the first layer's output for every
 * (centroid, neighbor) row:
 *   h1[b, c, k, :] = ReLU(P1[b, nit[b, c, k], :] - Q[b, c, :] + b1)
 * in fp64 on the stored fp32 tables, one rounding to fp32.  Layout:
 * p1 [B, N, C], q [B, M, C], b1 [C] (may be NULL), nit [B, M, K],
 * h1 [B, M, K, C].
 */
void orc_ltd_group(const float* p1, const float* q, const float* b1, const int32_t* nit, int64_t B, int64_t N,
                   int64_t M, int32_t K, int32_t C, float* h1) {
    for (int64_t b = 0; b < B; ++b)
        for (int64_t c = 0; c < M; ++c)
            for (int32_t k = 0; k < K; ++k) {
                const int64_t j = nit[(b * M + c) * K + k];
                const float* pr = p1 + (b * N + j) * C;
                const float* qr = q + (b * M + c) * C;
                float* out = h1 + ((b * M + c) * K + k) * C;
                for (int32_t ch = 0; ch < C; ++ch) {
                    double v = (double)pr[ch] - (double)qr[ch] + (b1 ? (double)b1[ch] : 0.0);
                    out[ch] = (float)(v > 0.0 ? v : 0.0);
                }
            }
}

/* Reduction after F in the conventional module (Sec. 3.1, last paragraph of
 * "Feature Computation"): column-wise max over each group of G rows. */
void orc_rowgroup_max(const float* y, int64_t groups, int32_t G, int32_t C, float* out, int64_t ld_out) {
    for (int64_t g = 0; g < groups; ++g)
        for (int32_t c = 0; c < C; ++c) {
            float mx = y[(g * G) * C + c];
            for (int32_t r = 1; r < G; ++r) {
                float v = y[(g * G + r) * C + c];
                if (v > mx) mx = v;
            }
            out[g * ld_out + c] = mx;
        }
}

/* ------------------------------------------------------------------------
 * Feature propagation by 3-NN inverse-distance interpolation
 * (three_interpolate of the PointNet++ segmentation baseline, Sec. 6,
 * Software Setup).  Weights 1 / max(d2, 1e-10) over the 3 nearest source
 * points (by orc_knn's rule), normalised; arithmetic in fp64, one final
 * rounding to fp32.
 * ---------------------------------------------------------------------- */
void orc_interpolate3(const float* xyz_dst, const float* xyz_src, const float* f_src, int64_t ld_src,
                      int64_t B, int64_t Nd, int64_t Ns, int32_t C, float* f_dst, int64_t ld_dst) {
    int32_t nn[3];
    float dd[3];
    for (int64_t b = 0; b < B; ++b)
        for (int64_t i = 0; i < Nd; ++i) {
            orc_knn(xyz_src + b * Ns * 3, 3, xyz_dst + (b * Nd + i) * 3, 3, 1, Ns, 1, 3, 3, nn, dd);
            double w[3], wsum = 0.0;
            for (int k = 0; k < 3; ++k) {
                double d = (double)dd[k];
                if (d < 1e-10) d = 1e-10;
                w[k] = 1.0 / d;
                wsum += w[k];
            }
            for (int32_t c = 0; c < C; ++c) {
                double acc = 0.0;
                for (int k = 0; k < 3; ++k) acc += w[k] * (double)f_src[(b * Ns + nn[k]) * ld_src + c];
                f_dst[(b * Nd + i) * ld_dst + c] = (float)(acc / wsum);
            }
        }
}

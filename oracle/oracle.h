/*
 * CPU oracle for delayed-aggregation point-cloud modules.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path links, loads or
 * calls this library; it exists so that tests, the smoke check and the
 * CPU-baseline leg of the benchmark can check the HIP path against a plain,
 * slow, obviously correct implementation.  It shares no code, header,
 * table or helper with the HIP library.
 *
 * Paper: Feng et al., "Mesorasi: Architecture Support for Point Cloud
 * Analytics via Delayed-Aggregation" (MICRO 2020, arXiv 2008.06967).
 *
 * Conventions (readings where the paper is silent; each one is listed in
 * the design notes of the repository):
 *  - dist2(a, b, C): t_c = a_c - b_c, d <- fma(t_c, t_c, d) for c ascending,
 *    starting from d = 0, every step rounded to fp32.  Symmetric in (a, b).
 *  - FPS starts at index 0, uses squared distances and breaks argmax ties
 *    towards the lowest index.
 *  - Ball query keeps the first K indices (ascending) with dist2 < r*r
 *    (r*r rounded to fp32) and pads with the first hit (0 when none).
 *  - kNN orders candidates by (dist2, index), self included.
 *  - MLP layers accumulate x_i * W[o][i] for i ascending in fp64, add the
 *    bias, round to fp32, apply ReLU (v > 0 ? v : +0) when the layer's bit
 *    is set in relu_mask.  bf16 mode rounds inputs and weights to bf16
 *    (round-to-nearest-even) and rounds every stored activation to bf16.
 *  - Aggregation: max over the K gathered rows (strict '>' keeps the earlier
 *    value), then one fp32 add/subtract of the centroid row.
 *
 * All index arrays are int32 and local to their cloud (0 <= i < N).
 */
#ifndef MESORASI_ORACLE_H
#define MESORASI_ORACLE_H
#include <stdint.h>

float orc_dist2(const float* a, const float* b, int C);
float orc_bf16_round(float f);

void orc_fps(const float* xyz, int64_t B, int64_t N, int64_t M, int32_t* idx, float* cxyz);
void orc_fps_bruteforce(const float* xyz, int64_t B, int64_t N, int64_t M, int32_t* idx);

void orc_ball_query(const float* xyz, const float* qxyz, int64_t B, int64_t N, int64_t M, float radius,
                    int32_t K, int32_t* nit, int32_t* cnt, int64_t* scanned);

void orc_knn(const float* ref, int64_t ld_ref, const float* query, int64_t ld_query, int64_t B, int64_t N,
             int64_t M, int32_t C, int32_t K, int32_t* nit, float* dist);

void orc_mlp(const float* x, int64_t rows, int32_t n_layers, const int32_t* dims, const float* const* W,
             const float* const* bias, uint32_t relu_mask, int32_t bf16, float* y);

void orc_aggregate_max(const float* pft, int64_t ld_pft, const int32_t* nit, int64_t B, int64_t N, int64_t M,
                       int32_t K, int32_t C, const int32_t* cidx, const float* cfeat, int64_t ld_c,
                       int32_t sign, int32_t relu, float* out, int64_t ld_out);

void orc_group_pointnet(const float* xyz, const float* feat, int32_t cf, int64_t ld_f, const float* cxyz,
                        const int32_t* nit, int64_t B, int64_t N, int64_t M, int32_t K, float* nfm);
void orc_group_offsets(const float* xyz, const float* feat, int32_t cf, int64_t ld_f, const int32_t* cidx,
                       const int32_t* nit, int64_t B, int64_t N, int64_t M, int32_t K, float* nfm);
void orc_group_edge(const float* f, int64_t ld_f, int32_t C, const int32_t* nit, int64_t B, int64_t N,
                    int32_t K, float* nfm);

void orc_rowgroup_max(const float* y, int64_t groups, int32_t G, int32_t C, float* out, int64_t ld_out);

void orc_ltd_group(const float* p1, const float* q, const float* b1, const int32_t* nit, int64_t B, int64_t N,
                   int64_t M, int32_t K, int32_t C, float* h1);

void orc_interpolate3(const float* xyz_dst, const float* xyz_src, const float* f_src, int64_t ld_src,
                      int64_t B, int64_t Nd, int64_t Ns, int32_t C, float* f_dst, int64_t ld_dst);

#endif

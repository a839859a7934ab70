// Internal interface between the per-layer GEMM MLP (mlp.hip) and the fused
// narrow-layer MLP (mlp_fused.hip).
#pragma once

#include "common.h"

namespace meso {

// Rows of a gathered first layer, read straight from the inputs instead of
// a materialized (centroid, neighbor) matrix.  Row r = (cloud b, centroid
// c, neighbor k), r = (b M + c) K + k, belongs to point j = nit[r] of cloud
// b and is
//   q == null (conventional, PointNet++ grouping): [xyz_j - cxyz_c | feat_j]
//   q != null (limited order): ReLU((p1_j - q_c) + b1), p1 = the x0 rows.
struct MlpGather {
    const int32_t* nit;   // [B * M * K]
    int64_t mk;           // rows per cloud (M * K)
    int64_t n;            // points per cloud
    int k;                // rows per centroid
    const float* cxyz;    // [B * M, 3]
    const float* q;       // [B * M, ldq]
    int64_t ldq;
    const float* b1;      // nullable
};

// Rows of an aggregated first layer (the previous module's aggregation
// done in the loader): row r = (cloud b, centroid c), r = b M + c, is
// [cxyz_r | max_k pft[b, nit[r, k]] - pft[b, cidx[r]]] over C channels.
struct MlpAggregate {
    const float* pft;     // [B, n, ld_pft]
    int64_t ld_pft;
    int64_t n;            // points per cloud of the PFT
    int64_t m;            // centroids per cloud
    const int32_t* nit;   // [B * m, k]
    const int32_t* cidx;  // [B * m]
    int k;
    int C;
    float* out;           // nullable: the aggregated rows [B * m, ld_out]
    int64_t ld_out;
};

// True when every layer input fits the fused kernel's LDS tile.
bool fused_mlp_supported(int n_layers, const int32_t* dims, int dtype);

// Whole MLP in one launch (no workspace).  pool_group > 0 zero-fills y first.
int run_fused_mlp(const float* x0, int c0, int64_t ld0, const float* x1, int c1, int64_t ld1, int64_t rows,
                  int n_layers, const int32_t* dims, const void* const* W, const float* const* bias,
                  uint32_t relu_mask, int out_dtype, void* y, int64_t ld_y, int64_t pool_group, hipStream_t s,
                  const MlpGather* g = nullptr);

// True when every layer is at most 128 wide (the register-resident MLP,
// mlp_rr.hip) and either the permuted weights of all layers fit the LDS of
// one workgroup, or each fits and the rows make at most one 32-row tile
// per wave (the weights are then staged in phases).
bool rr_mlp_supported(int n_layers, const int32_t* dims, int64_t rows);

// First-layer rows made by interpolation (mesorasi_interpolate3_mlp): row r
// = b nd + i is phi(sum_k u_k g[b, nit[r, k]] + add[r]); every row and
// pointer 16-byte aligned, dims[0] % 4 == 0.
struct RrInterp {
    const int32_t* nit;   // [rows, 3]
    const float* dist;    // [rows, 3]
    const float* g;       // [B, ns, ldg]
    int64_t ldg, nd, ns;
    const float* add;     // [rows, lda]
    int64_t lda;
    int relu;
};

// The register-resident MLP: fp32 rows [x0 | x1] (or interpolated rows) in,
// fp32 y out, no workspace, no pooling.
int run_rr_mlp(const float* x0, int c0, int64_t ld0, const float* x1, int c1, int64_t ld1, int64_t rows,
               int n_layers, const int32_t* dims, const void* const* W, const float* const* bias,
               uint32_t relu_mask, float* y, int64_t ld_y, hipStream_t s, const RrInterp* ip = nullptr);

// The same for bf16 MLPs (mlp_rr_bf16.hip): every layer at most 128 wide;
// fp32 rows in, fp32 or bf16 y out (bf16-rounded values either way).
bool rb_mlp_supported(int n_layers, const int32_t* dims);
int run_rb_mlp(const float* x0, int c0, int64_t ld0, const float* x1, int c1, int64_t ld1, int64_t rows,
               int n_layers, const int32_t* dims, const void* const* W, const float* const* bias,
               uint32_t relu_mask, int out_dtype, void* y, int64_t ld_y, hipStream_t s);

// The aggregated-rows form of the fused MLP (fp32 in and out).
int run_fused_aggregate_mlp(const float* cxyz, const MlpAggregate& ag, int64_t rows, int n_layers,
                            const int32_t* dims, const void* const* W, const float* const* bias, uint32_t relu_mask,
                            float* y, int64_t ld_y, hipStream_t s);

}  // namespace meso

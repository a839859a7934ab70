// Internal interface between the per-layer GEMM MLP (mlp.hip) and the fused
// narrow-layer MLP (mlp_fused.hip).
#pragma once

#include "common.h"

namespace meso {

// True when every layer input fits the fused kernel's LDS tile.
bool fused_mlp_supported(int n_layers, const int32_t* dims, int dtype);

// Whole MLP in one launch (no workspace).  pool_group > 0 zero-fills y first.
int run_fused_mlp(const float* x0, int c0, int64_t ld0, const float* x1, int c1, int64_t ld1, int64_t rows,
                  int n_layers, const int32_t* dims, const void* const* W, const float* const* bias,
                  uint32_t relu_mask, int out_dtype, void* y, int64_t ld_y, int64_t pool_group, hipStream_t s);

}  // namespace meso

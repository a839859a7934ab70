// Internal helpers shared by the gfx950 kernels and the host launchers of
// libmesorasi.so.  Not part of the public ABI (include/mesorasi.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mesorasi.h"

namespace meso {

// ---------------------------------------------------------------------------
// host-side error state (thread-local text for mesorasi_last_error)
// ---------------------------------------------------------------------------
int set_error(int status, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int after_launch(const char* what);

#define MESO_REQUIRE(cond, status, ...)                  \
    do {                                                 \
        if (!(cond)) return ::meso::set_error(status, __VA_ARGS__); \
    } while (0)

inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

inline bool aligned(const void* p, int bytes) { return (reinterpret_cast<uintptr_t>(p) % bytes) == 0; }

// Zero-fill of a strided [rows, cols] float32 region (used before pooled
// atomics; a kernel rather than hipMemsetAsync so the call stays
// graph-capturable).
int zero_rows_f32(float* y, int64_t rows, int64_t cols, int64_t ld, hipStream_t s);

// ---------------------------------------------------------------------------
// device helpers
// ---------------------------------------------------------------------------

// Squared Euclidean distance in 3-D: t = a - b per axis, d = t_x^2,
// d = fma(t_y, t_y, d), d = fma(t_z, t_z, d).  Built with
// -ffp-contract=off, so the multiply and the two fmas are the only
// roundings.
__device__ __forceinline__ float dist3(float ax, float ay, float az, float bx, float by, float bz) {
    const float tx = ax - bx;
    const float ty = ay - by;
    const float tz = az - bz;
    float d = tx * tx;
    d = __builtin_fmaf(ty, ty, d);
    d = __builtin_fmaf(tz, tz, d);
    return d;
}

// float32 -> bf16 bits, round to nearest even (finite inputs).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7fffu + ((u >> 16) & 1u);
    return static_cast<uint16_t>(u >> 16);
}

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float(static_cast<uint32_t>(h) << 16); }

// Round a float to the nearest bf16 value, kept in float.
__device__ __forceinline__ float round_bf16(float f) { return bf16_to_f32(f32_to_bf16(f)); }

__device__ __forceinline__ int lane_id() { return __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u)); }

// Number of set bits of a wave mask below this lane.
__device__ __forceinline__ int mask_rank(uint64_t m) {
    return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(m >> 32),
                                     __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(m), 0u));
}

__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }

// v = max(v, dpp(v)) as one v_max_i32_dpp (bound_ctrl lets the compiler fuse
// the move into the max).
template <int CTRL>
__device__ __forceinline__ int dpp_max_i32(int v) {
    return max(v, __builtin_amdgcn_mov_dpp(v, CTRL, 0xf, 0xf, true));
}

// Max over the lanes of each 16-lane row, returned in every lane of the row
// (butterfly of row rotations).
__device__ __forceinline__ int row_max_i32(int v) {
    v = dpp_max_i32<0x121>(v);  // row_ror:1
    v = dpp_max_i32<0x122>(v);  // row_ror:2
    v = dpp_max_i32<0x124>(v);  // row_ror:4
    v = dpp_max_i32<0x128>(v);  // row_ror:8
    return v;
}

// Max over each group of 4 lanes, in every lane of the group.
__device__ __forceinline__ int quad_max_i32(int v) {
    v = dpp_max_i32<0xB1>(v);   // quad_perm [1,0,3,2]
    v = dpp_max_i32<0x4E>(v);   // quad_perm [2,3,0,1]
    return v;
}

// Max over each group of 8 lanes; lane 8g+7 holds the max of lanes 8g..8g+7.
__device__ __forceinline__ int oct_max_i32(int v) {
    v = dpp_max_i32<0x121>(v);  // row_ror:1
    v = dpp_max_i32<0x122>(v);  // row_ror:2
    v = dpp_max_i32<0x124>(v);  // row_ror:4
    return v;
}

// Max of a signed int over the wave, returned to every lane (uniform): row
// butterfly, then the GFX9 row broadcasts fold rows 0..3 into lane 63.
__device__ __forceinline__ int wave_max_i32(int v) {
    v = row_max_i32(v);
    v = max(v, __builtin_amdgcn_update_dpp(v, v, 0x142, 0xa, 0xf, false));  // row_bcast:15 into rows 1, 3
    v = max(v, __builtin_amdgcn_update_dpp(v, v, 0x143, 0xc, 0xf, false));  // row_bcast:31 into rows 2, 3
    return __builtin_amdgcn_readlane(v, 63);
}

}  // namespace meso

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

template <int CTRL>
__device__ __forceinline__ int dpp_i32(int v) {
    return __builtin_amdgcn_update_dpp(v, v, CTRL, 0xf, 0xf, false);
}

// Max of a signed int over the wave, returned to every lane.  Row-level
// butterfly with DPP row rotations (every lane of a 16-lane row ends with
// the row max), then the four row maxima are combined through readlane.
__device__ __forceinline__ int wave_max_i32(int v) {
    v = max(v, dpp_i32<0x121>(v));  // row_ror:1
    v = max(v, dpp_i32<0x122>(v));  // row_ror:2
    v = max(v, dpp_i32<0x124>(v));  // row_ror:4
    v = max(v, dpp_i32<0x128>(v));  // row_ror:8
    const int a = __builtin_amdgcn_readlane(v, 0);
    const int b = __builtin_amdgcn_readlane(v, 16);
    const int c = __builtin_amdgcn_readlane(v, 32);
    const int d = __builtin_amdgcn_readlane(v, 48);
    return max(max(a, b), max(c, d));
}

// Max over the lanes of one 16-lane row (row-local result in every lane).
__device__ __forceinline__ int row_max_i32(int v) {
    v = max(v, dpp_i32<0x121>(v));
    v = max(v, dpp_i32<0x122>(v));
    v = max(v, dpp_i32<0x124>(v));
    v = max(v, dpp_i32<0x128>(v));
    return v;
}

}  // namespace meso

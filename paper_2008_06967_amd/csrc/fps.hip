// Farthest-point sampling on gfx950: one workgroup per cloud.
//
// The sampling step of the PointNet++ modules (Sec. 5, "Software Setup")
// read as greedy max-min sampling from point 0, lowest index on ties.
//
// Layout: thread t of a T-thread workgroup owns the P consecutive points
// [t*P, t*P + P); their coordinates and running min-distances live in
// registers for the whole kernel (P <= 16), so an iteration reads no
// memory except one LDS exchange.  Because ownership is contiguous, "lowest
// index" = lowest point slot within a thread, then lowest lane within a
// wave, then lowest wave -- so every reduction below is a plain max on the
// distance bits (non-negative floats order like signed ints) followed by a
// "first lane holding the max" ballot.
//
// One barrier per iteration: the per-wave winners go to a double-buffered
// LDS slot array indexed by iteration parity, so a wave that runs ahead
// writes the other buffer while slower waves still read this one.
#include "common.h"

namespace meso {

template <int T, int P, bool REG_XYZ>
__global__ __launch_bounds__(T) void fps_kernel(const float* __restrict__ xyz, int N, int M, int32_t* __restrict__ idx,
                                                float* __restrict__ cxyz) {
    constexpr int W = T / 64;
    __shared__ int s_d[2][W];
    __shared__ int s_i[2][W];
    __shared__ float s_x[2][W];
    __shared__ float s_y[2][W];
    __shared__ float s_z[2][W];

    const int b = blockIdx.x;
    const float* __restrict__ p = xyz + (int64_t)b * N * 3;
    int32_t* __restrict__ out_idx = idx + (int64_t)b * M;
    float* __restrict__ out_c = cxyz ? cxyz + (int64_t)b * M * 3 : nullptr;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int base = tid * P;

    float px[REG_XYZ ? P : 1], py[REG_XYZ ? P : 1], pz[REG_XYZ ? P : 1];
    float dm[P];
#pragma unroll
    for (int q = 0; q < P; ++q) {
        const int j = base + q;
        const bool ok = j < N;
        if constexpr (REG_XYZ) {
            px[q] = ok ? p[3 * j + 0] : 0.0f;
            py[q] = ok ? p[3 * j + 1] : 0.0f;
            pz[q] = ok ? p[3 * j + 2] : 0.0f;
        }
        dm[q] = ok ? __builtin_huge_valf() : -1.0f;  // +inf for real points; -1 never wins
    }

    float cx = p[0], cy = p[1], cz = p[2];
    if (tid == 0) {
        out_idx[0] = 0;
        if (out_c) {
            out_c[0] = cx;
            out_c[1] = cy;
            out_c[2] = cz;
        }
    }

    for (int m = 1; m < M; ++m) {
        int bestd = __float_as_int(-1.0f);
        int bestq = 0;
        float bx = 0.0f, by = 0.0f, bz = 0.0f;
#pragma unroll
        for (int q = 0; q < P; ++q) {
            float x, y, z;
            if constexpr (REG_XYZ) {
                x = px[q];
                y = py[q];
                z = pz[q];
            } else {
                const int j = min(base + q, N - 1);
                x = p[3 * j + 0];
                y = p[3 * j + 1];
                z = p[3 * j + 2];
            }
            const float d = dist3(x, y, z, cx, cy, cz);
            const float nm = fminf(dm[q], d);
            dm[q] = nm;
            const int nb = __float_as_int(nm);
            if (nb > bestd) {
                bestd = nb;
                bestq = q;
                bx = x;
                by = y;
                bz = z;
            }
        }
        // wave winner: max distance, lowest lane among equals
        const int wmax = wave_max_i32(bestd);
        const uint64_t hit = ballot(bestd == wmax);
        const int wl = __builtin_ctzll(hit);
        const int buf = m & 1;
        if (lane == wl) {
            s_d[buf][wave] = wmax;
            s_i[buf][wave] = base + bestq;
            s_x[buf][wave] = bx;
            s_y[buf][wave] = by;
            s_z[buf][wave] = bz;
        }
        __syncthreads();
        // block winner: lane w < W inspects wave w's slot
        int vd = INT32_MIN;  // below every slot value (slots hold >= bits(-1.0f))
        int vi = 0;
        float vx = 0.0f, vy = 0.0f, vz = 0.0f;
        if (lane < W) {
            vd = s_d[buf][lane];
            vi = s_i[buf][lane];
            vx = s_x[buf][lane];
            vy = s_y[buf][lane];
            vz = s_z[buf][lane];
        }
        const int gmax = (W <= 16) ? __builtin_amdgcn_readlane(row_max_i32(vd), 0) : wave_max_i32(vd);
        const int ww = __builtin_ctzll(ballot(vd == gmax));
        const int sel = __builtin_amdgcn_readlane(vi, ww);
        cx = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(vx), ww));
        cy = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(vy), ww));
        cz = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(vz), ww));
        if (tid == 0) {
            out_idx[m] = sel;
            if (out_c) {
                out_c[3 * m + 0] = cx;
                out_c[3 * m + 1] = cy;
                out_c[3 * m + 2] = cz;
            }
        }
    }
}

template <int T, int P, bool REG>
static void launch_fps(const float* xyz, int64_t B, int N, int M, int32_t* idx, float* cxyz, hipStream_t s) {
    fps_kernel<T, P, REG><<<dim3((unsigned)B), dim3(T), 0, s>>>(xyz, N, M, idx, cxyz);
}

}  // namespace meso

using namespace meso;

extern "C" int mesorasi_fps(const float* xyz, int64_t B, int64_t N, int64_t M, int32_t* idx, float* cxyz,
                            void* stream) {
    MESO_REQUIRE(B >= 0 && N >= 0 && M >= 0, MESORASI_EINVAL, "mesorasi_fps: negative size (B=%lld N=%lld M=%lld)",
                 (long long)B, (long long)N, (long long)M);
    MESO_REQUIRE(M <= N, MESORASI_EINVAL, "mesorasi_fps: M = %lld > N = %lld", (long long)M, (long long)N);
    if (B == 0 || M == 0) return MESORASI_OK;
    MESO_REQUIRE(xyz && idx, MESORASI_EINVAL, "mesorasi_fps: NULL xyz or idx");
    MESO_REQUIRE(N <= MESORASI_MAX_N_FPS, MESORASI_EUNSUPPORTED, "mesorasi_fps: N = %lld > %d", (long long)N,
                 MESORASI_MAX_N_FPS);
    MESO_REQUIRE(B <= 0x7fffffff, MESORASI_EUNSUPPORTED, "mesorasi_fps: B too large");
    hipStream_t s = as_stream(stream);
    const int n = (int)N, m = (int)M;
    if (n <= 64) launch_fps<64, 1, true>(xyz, B, n, m, idx, cxyz, s);
    else if (n <= 128) launch_fps<64, 2, true>(xyz, B, n, m, idx, cxyz, s);
    else if (n <= 256) launch_fps<128, 2, true>(xyz, B, n, m, idx, cxyz, s);
    else if (n <= 512) launch_fps<256, 2, true>(xyz, B, n, m, idx, cxyz, s);
    else if (n <= 1024) launch_fps<256, 4, true>(xyz, B, n, m, idx, cxyz, s);
    else if (n <= 2048) launch_fps<512, 4, true>(xyz, B, n, m, idx, cxyz, s);
    else if (n <= 4096) launch_fps<1024, 4, true>(xyz, B, n, m, idx, cxyz, s);
    else if (n <= 8192) launch_fps<1024, 8, true>(xyz, B, n, m, idx, cxyz, s);
    else if (n <= 16384) launch_fps<1024, 16, true>(xyz, B, n, m, idx, cxyz, s);
    else if (n <= 32768) launch_fps<1024, 32, false>(xyz, B, n, m, idx, cxyz, s);
    else launch_fps<1024, 64, false>(xyz, B, n, m, idx, cxyz, s);
    return after_launch("mesorasi_fps");
}

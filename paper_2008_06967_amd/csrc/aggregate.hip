// Aggregation on the point feature table, gfx950.
//
// Sec. 5.2 (first paragraph): for every NIT entry gather the K PFT rows,
// reduce them column-wise with max, then combine with the centroid's row
// (max(f_j - f_c) = max(f_j) - f_c, end of the Sec. 4.1 walk-through).
//
// Mapping: one wave per (centroid, channel slice).  A lane loads 16 bytes
// of a row (4 fp32 or 8 bf16 channels); LPR lanes cover a row slice of
// LPR*VEC channels, so one wave-wide load fetches RPW = 64/LPR neighbor rows
// at once (a C = 128 fp32 PFT: 32 lanes per row, 2 rows per load).  The
// centroid's NIT row is read once (one index per lane) and distributed by
// cross-lane reads, so eight row gathers per lane are in flight at a time.
// The running max lives in registers; the RPW partial maxima are folded
// with cross-lane max at the end and one fp32 add/subtract applies the
// centroid row.  Workgroups are renumbered so that each XCD's L2 serves a
// contiguous range of clouds.  Nothing N x K x C sized is ever written.  Wider PFTs are split into
// channel slices processed by different waves -- the column partitioning
// of the paper's PFT buffer (Sec. 5.2, "PFT Partitioning").
#include "common.h"

namespace meso {

template <typename T>
__device__ __forceinline__ float to_f32(T v);
template <>
__device__ __forceinline__ float to_f32<float>(float v) {
    return v;
}
template <>
__device__ __forceinline__ float to_f32<uint16_t>(uint16_t v) {
    return bf16_to_f32(v);
}

// Load VEC consecutive elements starting at p, widened to float.
template <typename T, int VEC>
__device__ __forceinline__ void load_vec(const T* __restrict__ p, float (&v)[VEC]) {
    if constexpr (VEC == 1) {
        v[0] = to_f32<T>(p[0]);
    } else if constexpr (sizeof(T) == 4) {
        const float4 q = *reinterpret_cast<const float4*>(p);
        v[0] = q.x;
        v[1] = q.y;
        v[2] = q.z;
        v[3] = q.w;
    } else {
        const uint4 q = *reinterpret_cast<const uint4*>(p);
        const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            v[2 * i] = __uint_as_float(w[i] << 16);
            v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
        }
    }
}

template <typename T, int VEC, int LPR>
__global__ __launch_bounds__(256) void aggregate_kernel(const T* __restrict__ pft, int64_t ldp,
                                                        const int32_t* __restrict__ nit, int N, int M, int K, int C,
                                                        int chunks, int64_t total_waves, int per_xcd,
                                                        const int32_t* __restrict__ cidx,
                                                        const T* __restrict__ cfeat, int64_t ldc, int sign, int relu,
                                                        float* __restrict__ out, int64_t ldo) {
    constexpr int RPW = 64 / LPR;
    constexpr int CPW = LPR * VEC;
    constexpr int U = 8;   // row loads in flight per lane
    // Workgroups are dealt to the 8 XCDs round-robin by id; renumber them so
    // each XCD runs one contiguous range of centroids (hence whole clouds),
    // keeping a cloud's PFT rows in that XCD's L2.
    const int64_t lb = (int64_t)(blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
    const int64_t gw = lb * 4 + (threadIdx.x >> 6);
    if (gw >= total_waves) return;
    const int lane = threadIdx.x & 63;
    const int64_t c = gw / chunks;              // global centroid index in [0, B*M)
    const int chunk = (int)(gw - c * chunks);
    const int64_t b = c / M;
    const int sub = lane / LPR;
    const int ch0 = chunk * CPW + (lane % LPR) * VEC;
    const bool active = ch0 < C;
    const int32_t* __restrict__ nrow = nit + c * K;
    const T* __restrict__ cloud = pft + b * (int64_t)N * ldp + ch0;

    float mx[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) mx[v] = -__builtin_huge_valf();

    for (int kb = 0; kb < K; kb += 64) {
        // lane l holds neighbor kb + l of this centroid; rows are then
        // addressed through cross-lane reads, so all gathers issue together
        const int kn = min(64, K - kb);
        const int jreg = lane < kn ? nrow[kb + lane] : 0;
        const int nt = (kn + RPW - 1) / RPW;
        int t = 0;
        for (; t + U <= nt; t += U) {
            float a[U][VEC];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int k = sub + RPW * (t + u);
                const int j = __shfl(jreg, k < kn ? k : 0);
                if (active && k < kn) {
                    load_vec<T, VEC>(cloud + (int64_t)j * ldp, a[u]);
                } else {
#pragma unroll
                    for (int v = 0; v < VEC; ++v) a[u][v] = -__builtin_huge_valf();
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
                for (int v = 0; v < VEC; ++v) mx[v] = fmaxf(mx[v], a[u][v]);
        }
        for (; t < nt; ++t) {
            const int k = sub + RPW * t;
            const int j = __shfl(jreg, k < kn ? k : 0);
            if (active && k < kn) {
                float a[VEC];
                load_vec<T, VEC>(cloud + (int64_t)j * ldp, a);
#pragma unroll
                for (int v = 0; v < VEC; ++v) mx[v] = fmaxf(mx[v], a[v]);
            }
        }
    }
    // fold the RPW row slots (lanes l, l + LPR, l + 2 LPR, ...)
#pragma unroll
    for (int off = LPR; off < 64; off <<= 1) {
#pragma unroll
        for (int v = 0; v < VEC; ++v) mx[v] = fmaxf(mx[v], __shfl_xor(mx[v], off));
    }
    if (sub != 0 || !active) return;
    float r[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) r[v] = mx[v];
    if (cidx || cfeat) {
        float cen[VEC];
        if (cidx) load_vec<T, VEC>(cloud + (int64_t)cidx[c] * ldp, cen);
        else load_vec<T, VEC>(cfeat + c * ldc + ch0, cen);
#pragma unroll
        for (int v = 0; v < VEC; ++v) r[v] = sign < 0 ? mx[v] - cen[v] : mx[v] + cen[v];
    }
    if (relu) {
#pragma unroll
        for (int v = 0; v < VEC; ++v) r[v] = r[v] > 0.0f ? r[v] : 0.0f;
    }
    float* __restrict__ o = out + c * ldo + ch0;
    if constexpr (VEC == 1) {
        o[0] = r[0];
    } else if constexpr (VEC == 4) {
        *reinterpret_cast<float4*>(o) = make_float4(r[0], r[1], r[2], r[3]);
    } else {
        *reinterpret_cast<float4*>(o) = make_float4(r[0], r[1], r[2], r[3]);
        *reinterpret_cast<float4*>(o + 4) = make_float4(r[4], r[5], r[6], r[7]);
    }
}

template <typename T, int VEC>
static void launch_aggregate(const T* pft, int64_t ldp, const int32_t* nit, int64_t B, int N, int M, int K, int C,
                             const int32_t* cidx, const T* cfeat, int64_t ldc, int sign, int relu, float* out,
                             int64_t ldo, hipStream_t s) {
    const int lanes_needed = (C + VEC - 1) / VEC;
    int lpr = 1;
    while (lpr < lanes_needed && lpr < 64) lpr <<= 1;
    const int chunks = (C + lpr * VEC - 1) / (lpr * VEC);
    const int64_t total = B * (int64_t)M * chunks;
    const int64_t logical_blocks = ceil_div(total, 4);
    const int per_xcd = (int)ceil_div(logical_blocks, 8);
    const dim3 grid((unsigned)(8 * (int64_t)per_xcd)), block(256);
#define MESO_AGG_CASE(L)                                                                                          \
    case L:                                                                                                       \
        aggregate_kernel<T, VEC, L><<<grid, block, 0, s>>>(pft, ldp, nit, N, M, K, C, chunks, total, per_xcd, cidx, \
                                                           cfeat, ldc, sign, relu, out, ldo);                     \
        break;
    switch (lpr) {
        MESO_AGG_CASE(1)
        MESO_AGG_CASE(2)
        MESO_AGG_CASE(4)
        MESO_AGG_CASE(8)
        MESO_AGG_CASE(16)
        MESO_AGG_CASE(32)
        MESO_AGG_CASE(64)
    }
#undef MESO_AGG_CASE
}

}  // namespace meso

using namespace meso;

extern "C" int mesorasi_aggregate_max(const void* pft, int64_t ld_pft, int32_t pft_dtype, const int32_t* nit,
                                      int64_t B, int64_t N, int64_t M, int32_t K, int32_t C, const int32_t* cidx,
                                      const void* cfeat, int64_t ld_c, int32_t sign, int32_t relu, float* out,
                                      int64_t ld_out, void* stream) {
    MESO_REQUIRE(B >= 0 && N >= 0 && M >= 0, MESORASI_EINVAL, "mesorasi_aggregate_max: negative size");
    MESO_REQUIRE(K >= 1 && C >= 1, MESORASI_EINVAL, "mesorasi_aggregate_max: K = %d, C = %d", K, C);
    MESO_REQUIRE(ld_pft >= C && ld_out >= C, MESORASI_EINVAL, "mesorasi_aggregate_max: leading dimension < C");
    MESO_REQUIRE(!(cidx && cfeat), MESORASI_EINVAL, "mesorasi_aggregate_max: both cidx and cfeat given");
    MESO_REQUIRE(!cfeat || ld_c >= C, MESORASI_EINVAL, "mesorasi_aggregate_max: ld_c < C");
    MESO_REQUIRE(sign == 1 || sign == -1, MESORASI_EINVAL, "mesorasi_aggregate_max: sign = %d", sign);
    MESO_REQUIRE(pft_dtype == MESORASI_F32 || pft_dtype == MESORASI_BF16, MESORASI_EUNSUPPORTED,
                 "mesorasi_aggregate_max: dtype %d", pft_dtype);
    MESO_REQUIRE(C <= 65536, MESORASI_EUNSUPPORTED, "mesorasi_aggregate_max: C = %d > 65536", C);
    if (B == 0 || M == 0) return MESORASI_OK;
    MESO_REQUIRE(N >= 1, MESORASI_EINVAL, "mesorasi_aggregate_max: N = 0 with M > 0");
    MESO_REQUIRE(pft && nit && out, MESORASI_EINVAL, "mesorasi_aggregate_max: NULL pft, nit or out");
    MESO_REQUIRE(N <= 0x7fffffff && M <= 0x7fffffff, MESORASI_EUNSUPPORTED, "mesorasi_aggregate_max: size");
    hipStream_t s = as_stream(stream);
    const int n = (int)N, m = (int)M;
    if (pft_dtype == MESORASI_F32) {
        const float* p = static_cast<const float*>(pft);
        const float* cf = static_cast<const float*>(cfeat);
        const bool vec = C % 4 == 0 && ld_pft % 4 == 0 && ld_out % 4 == 0 && aligned(p, 16) && aligned(out, 16) &&
                         (!cf || (ld_c % 4 == 0 && aligned(cf, 16)));
        if (vec) launch_aggregate<float, 4>(p, ld_pft, nit, B, n, m, K, C, cidx, cf, ld_c, sign, relu, out, ld_out, s);
        else launch_aggregate<float, 1>(p, ld_pft, nit, B, n, m, K, C, cidx, cf, ld_c, sign, relu, out, ld_out, s);
    } else {
        const uint16_t* p = static_cast<const uint16_t*>(pft);
        const uint16_t* cf = static_cast<const uint16_t*>(cfeat);
        const bool vec = C % 8 == 0 && ld_pft % 8 == 0 && ld_out % 4 == 0 && aligned(p, 16) && aligned(out, 16) &&
                         (!cf || (ld_c % 8 == 0 && aligned(cf, 16)));
        if (vec)
            launch_aggregate<uint16_t, 8>(p, ld_pft, nit, B, n, m, K, C, cidx, cf, ld_c, sign, relu, out, ld_out, s);
        else
            launch_aggregate<uint16_t, 1>(p, ld_pft, nit, B, n, m, K, C, cidx, cf, ld_c, sign, relu, out, ld_out, s);
    }
    return after_launch("mesorasi_aggregate_max");
}

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
//
// LDS form (aggregate_lds_kernel), used when a column slice of one cloud's
// PFT fits the 160 KB LDS and the batch gives enough workgroups: this is
// the paper's on-chip PFT buffer with its column partitioning (Sec. 5.2).
// A 1024-thread workgroup copies slice s (32 or 16 fp32 channels, 64 or 32
// bf16) of cloud b's PFT into LDS once, with coalesced 16-byte loads, then
// gathers every NIT row of its share of the cloud's centroids from LDS:
// lane (g, q) of a wave serves centroid g of the pass and 16 bytes q of
// the slice, so one LDS read instruction fetches 64 / Q neighbor rows of
// Q x 16 bytes.  Random-row LDS gathers run at ~117-139 B/clk per CU on
// gfx950 against ~32 B/clk for the same gathers through the vector L1, which
// is what bounds the L2 form at batch size.  Neighbor indices come straight
// from global memory four at a time (16-byte rows of the NIT).
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

// Slice widths in 16-byte units per row (Q) and the launch shape.
constexpr int kAggLdsThreads = 1024;
constexpr int kAggLdsMaxTile = 128 * 1024;   // tile bytes (the NIT stays in global memory)

template <typename T, int Q>
__global__ __launch_bounds__(kAggLdsThreads) void aggregate_lds_kernel(
    const T* __restrict__ pft, int64_t ldp, const int32_t* __restrict__ nit, int N, int M, int K, int C, int slices,
    int parts, int64_t nblocks, int per_xcd, const int32_t* __restrict__ cidx, const T* __restrict__ cfeat,
    int64_t ldc, int sign, int relu, float* __restrict__ out, int64_t ldo) {
    constexpr int VEC = 16 / sizeof(T);          // elements per 16 bytes
    constexpr int CS = Q * VEC;                  // channels per slice
    constexpr int G = 64 / Q;                    // centroids per wave pass
    constexpr int NW = kAggLdsThreads / 64;
    extern __shared__ uint4 tile[];              // [N][Q] 16-byte units
    // renumber so that each XCD runs one contiguous range of (cloud, slice, part)
    const int64_t lb = (int64_t)(blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
    if (lb >= nblocks) return;
    const int part = (int)(lb % parts);
    const int64_t bs = lb / parts;
    const int s = (int)(bs % slices);
    const int64_t b = bs / slices;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int ch0 = s * CS;

    // 1. the slice of the cloud's PFT into LDS (columns past C as zeros)
    const T* __restrict__ src = pft + b * (int64_t)N * ldp + ch0;
    constexpr int U = 8;
    const int total = N * Q;
    for (int i0 = 0; i0 < total; i0 += kAggLdsThreads * U) {
        uint4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int i = i0 + u * kAggLdsThreads + tid;
            const int r = i / Q, qq = i % Q;
            const bool ok = i < total && ch0 + qq * VEC < C;
            v[u] = ok ? *reinterpret_cast<const uint4*>(src + (int64_t)r * ldp + qq * VEC) : make_uint4(0u, 0u, 0u, 0u);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int i = i0 + u * kAggLdsThreads + tid;
            if (i < total) tile[i] = v[u];
        }
    }
    __syncthreads();

    // 2. this part's centroids, G per wave pass
    const int per = (M + parts - 1) / parts;
    const int cb = part * per, ce = min(M, cb + per);
    const int g = lane / Q, q = lane % Q;
    const bool chok = ch0 + q * VEC < C;
    const int K4 = K / 4;
    for (int c0 = cb + wave * G; c0 < ce; c0 += NW * G) {
        const int c = min(c0 + g, ce - 1);
        const int64_t gc = b * M + c;
        const int4* __restrict__ nr = reinterpret_cast<const int4*>(nit + gc * K);
        float mx[VEC];
#pragma unroll
        for (int v = 0; v < VEC; ++v) mx[v] = -__builtin_huge_valf();
        auto take = [&](int j) {
            const uint4 w = tile[j * Q + q];
            float a[VEC];
            if constexpr (sizeof(T) == 4) {
                a[0] = __uint_as_float(w.x); a[1] = __uint_as_float(w.y);
                a[2] = __uint_as_float(w.z); a[3] = __uint_as_float(w.w);
            } else {
                const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    a[2 * i] = __uint_as_float(ws[i] << 16);
                    a[2 * i + 1] = __uint_as_float(ws[i] & 0xffff0000u);
                }
            }
#pragma unroll
            for (int v = 0; v < VEC; ++v) mx[v] = fmaxf(mx[v], a[v]);
        };
        for (int k4 = 0; k4 < K4; k4 += 2) {
            const int4 ja = nr[k4];
            const int4 jb = nr[min(k4 + 1, K4 - 1)];   // a repeated row does not change the max
            take(ja.x); take(ja.y); take(ja.z); take(ja.w);
            take(jb.x); take(jb.y); take(jb.z); take(jb.w);
        }
        float cen[VEC];
        if (cidx) {
            const uint4 w = tile[cidx[gc] * Q + q];
            if constexpr (sizeof(T) == 4) {
                cen[0] = __uint_as_float(w.x); cen[1] = __uint_as_float(w.y);
                cen[2] = __uint_as_float(w.z); cen[3] = __uint_as_float(w.w);
            } else {
                const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    cen[2 * i] = __uint_as_float(ws[i] << 16);
                    cen[2 * i + 1] = __uint_as_float(ws[i] & 0xffff0000u);
                }
            }
        } else if (cfeat && chok) {
            load_vec<T, VEC>(cfeat + gc * ldc + ch0 + q * VEC, cen);
        }
        if (c0 + g >= ce || !chok) continue;
        float r[VEC];
#pragma unroll
        for (int v = 0; v < VEC; ++v) {
            r[v] = mx[v];
            if (cidx || cfeat) r[v] = sign < 0 ? mx[v] - cen[v] : mx[v] + cen[v];
            if (relu) r[v] = r[v] > 0.0f ? r[v] : 0.0f;
        }
        float* __restrict__ o = out + gc * ldo + ch0 + q * VEC;
#pragma unroll
        for (int v = 0; v < VEC; v += 4) *reinterpret_cast<float4*>(o + v) = make_float4(r[v], r[v + 1], r[v + 2], r[v + 3]);
    }
}

// LDS form plan: the widest slice (Q = 8, else 4) whose tile fits and
// that reaches 256 workgroups with at most 2 (Q = 8) or 4 (Q = 4) parts per
// slice, each part gathering at least twice the tile; none -> L2 form.
struct AggLdsPlan {
    int q, slices, parts;
};
static AggLdsPlan plan_aggregate_lds(int64_t B, int N, int M, int K, int C, int elem) {
    const int vec = 16 / elem;
    for (int q : {8, 4}) {
        if ((int64_t)N * q * 16 > kAggLdsMaxTile) continue;
        const int slices = (int)ceil_div(C, q * vec);
        int parts = 1;
        while (B * slices * parts < 256 && parts < 64) parts *= 2;
        if (parts > (q == 8 ? 2 : 4)) continue;
        const int64_t per = ceil_div(M, parts);
        if (per * K < 2 * (int64_t)N) continue;
        return {q, slices, parts};
    }
    return {0, 0, 0};
}

template <typename T, int Q>
static int launch_aggregate_lds(const T* pft, int64_t ldp, const int32_t* nit, int64_t B, int N, int M, int K, int C,
                                const AggLdsPlan& pl, const int32_t* cidx, const T* cfeat, int64_t ldc, int sign,
                                int relu, float* out, int64_t ldo, hipStream_t s) {
    static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(&aggregate_lds_kernel<T, Q>),
                                                       hipFuncAttributeMaxDynamicSharedMemorySize, kAggLdsMaxTile);
    MESO_REQUIRE(attr == hipSuccess, MESORASI_EHIP, "mesorasi_aggregate_max: LDS size attribute: %s",
                 hipGetErrorString(attr));
    const int64_t nb = B * pl.slices * pl.parts;
    const int per_xcd = (int)ceil_div(nb, 8);
    const size_t lds = (size_t)N * Q * 16;
    aggregate_lds_kernel<T, Q><<<dim3((unsigned)(8 * per_xcd)), dim3(kAggLdsThreads), lds, s>>>(
        pft, ldp, nit, N, M, K, C, pl.slices, pl.parts, nb, per_xcd, cidx, cfeat, ldc, sign, relu, out, ldo);
    return MESORASI_OK;
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
    // the LDS form reads NIT rows as 16-byte vectors
    const bool lds_ok = K % 4 == 0 && aligned(nit, 16);
    if (pft_dtype == MESORASI_F32) {
        const float* p = static_cast<const float*>(pft);
        const float* cf = static_cast<const float*>(cfeat);
        const bool vec = C % 4 == 0 && ld_pft % 4 == 0 && ld_out % 4 == 0 && aligned(p, 16) && aligned(out, 16) &&
                         (!cf || (ld_c % 4 == 0 && aligned(cf, 16)));
        const AggLdsPlan pl = vec && lds_ok ? plan_aggregate_lds(B, n, m, K, C, 4) : AggLdsPlan{0, 0, 0};
        if (pl.q == 8) {
            const int rc = launch_aggregate_lds<float, 8>(p, ld_pft, nit, B, n, m, K, C, pl, cidx, cf, ld_c, sign, relu,
                                                          out, ld_out, s);
            if (rc != MESORASI_OK) return rc;
        } else if (pl.q == 4) {
            const int rc = launch_aggregate_lds<float, 4>(p, ld_pft, nit, B, n, m, K, C, pl, cidx, cf, ld_c, sign, relu,
                                                          out, ld_out, s);
            if (rc != MESORASI_OK) return rc;
        } else if (vec) {
            launch_aggregate<float, 4>(p, ld_pft, nit, B, n, m, K, C, cidx, cf, ld_c, sign, relu, out, ld_out, s);
        } else {
            launch_aggregate<float, 1>(p, ld_pft, nit, B, n, m, K, C, cidx, cf, ld_c, sign, relu, out, ld_out, s);
        }
    } else {
        const uint16_t* p = static_cast<const uint16_t*>(pft);
        const uint16_t* cf = static_cast<const uint16_t*>(cfeat);
        const bool vec = C % 8 == 0 && ld_pft % 8 == 0 && ld_out % 4 == 0 && aligned(p, 16) && aligned(out, 16) &&
                         (!cf || (ld_c % 8 == 0 && aligned(cf, 16)));
        const AggLdsPlan pl = vec && lds_ok ? plan_aggregate_lds(B, n, m, K, C, 2) : AggLdsPlan{0, 0, 0};
        if (pl.q == 8) {
            const int rc = launch_aggregate_lds<uint16_t, 8>(p, ld_pft, nit, B, n, m, K, C, pl, cidx, cf, ld_c, sign,
                                                             relu, out, ld_out, s);
            if (rc != MESORASI_OK) return rc;
        } else if (pl.q == 4) {
            const int rc = launch_aggregate_lds<uint16_t, 4>(p, ld_pft, nit, B, n, m, K, C, pl, cidx, cf, ld_c, sign,
                                                             relu, out, ld_out, s);
            if (rc != MESORASI_OK) return rc;
        } else if (vec) {
            launch_aggregate<uint16_t, 8>(p, ld_pft, nit, B, n, m, K, C, cidx, cf, ld_c, sign, relu, out, ld_out, s);
        } else {
            launch_aggregate<uint16_t, 1>(p, ld_pft, nit, B, n, m, K, C, cidx, cf, ld_c, sign, relu, out, ld_out, s);
        }
    }
    return after_launch("mesorasi_aggregate_max");
}

// Ball query on gfx950 -- the neighbor search N (Sec. 3.1 "Neighbor Search")
// that fills the neighbor index table (NIT, Sec. 4.1 walk-through).
//
// One wave per query.  The wave walks the cloud in 64-point chunks in index
// order (coordinates fetched four chunks at a time); each lane tests one point, a ballot collects the chunk's hits and
// mbcnt gives every hit its rank, so hits land in ascending index order with
// no sorting.  The walk stops as soon as K hits are found (the early exit is
// what makes surface-like clouds cheap), then the tail of the row is padded
// with the first hit.
#include "common.h"

namespace meso {

constexpr int kBqWaves = 4;
constexpr int kBqChunks = 4;   // 64-point chunks per memory round trip

__global__ __launch_bounds__(64 * kBqWaves) void ball_query_kernel(const float* __restrict__ xyz,
                                                                   const float* __restrict__ qxyz, int64_t BM, int N,
                                                                   int M, float r2, int K, int32_t* __restrict__ nit,
                                                                   int32_t* __restrict__ cnt) {
    const int64_t gq = (int64_t)blockIdx.x * kBqWaves + (threadIdx.x >> 6);
    if (gq >= BM) return;  // whole wave leaves together; no barriers below
    const int lane = threadIdx.x & 63;
    const int64_t b = gq / M;
    const float* __restrict__ p = xyz + b * (int64_t)N * 3;
    const float qx = qxyz[gq * 3 + 0], qy = qxyz[gq * 3 + 1], qz = qxyz[gq * 3 + 2];
    int32_t* __restrict__ row = nit + gq * K;

    int n = 0;
    int first = 0;
    for (int base0 = 0; base0 < N && n < K; base0 += 64 * kBqChunks) {
        // the coordinates of kBqChunks chunks are requested together (lanes
        // past N read point N - 1 and never hit), so one memory round trip
        // serves several chunks; the chunks are still tested in index order
        // and the walk stops after the chunk that completes K hits
        float cx[kBqChunks], cy[kBqChunks], cz[kBqChunks];
#pragma unroll
        for (int u = 0; u < kBqChunks; ++u) {
            const int64_t j = min(base0 + 64 * u + lane, N - 1);
            cx[u] = p[3 * j + 0];
            cy[u] = p[3 * j + 1];
            cz[u] = p[3 * j + 2];
        }
#pragma unroll
        for (int u = 0; u < kBqChunks; ++u) {
            const int base = base0 + 64 * u;
            if (base >= N || n >= K) break;
            const int j = base + lane;
            const bool hit = j < N && dist3(cx[u], cy[u], cz[u], qx, qy, qz) < r2;
            const uint64_t mask = ballot(hit);
            if (mask) {
                if (n == 0) first = base + __builtin_ctzll(mask);
                const int pos = n + mask_rank(mask);
                if (hit && pos < K) row[pos] = j;
                n += __builtin_popcountll(mask);
            }
        }
    }
    n = min(n, K);
    const int pad = n > 0 ? first : 0;
    for (int k = n + lane; k < K; k += 64) row[k] = pad;
    if (cnt && lane == 0) cnt[gq] = n;
}

}  // namespace meso

using namespace meso;

extern "C" int mesorasi_ball_query(const float* xyz, const float* qxyz, int64_t B, int64_t N, int64_t M,
                                   float radius, int32_t K, int32_t* nit, int32_t* cnt, void* stream) {
    MESO_REQUIRE(B >= 0 && N >= 0 && M >= 0, MESORASI_EINVAL, "mesorasi_ball_query: negative size");
    MESO_REQUIRE(K >= 1, MESORASI_EINVAL, "mesorasi_ball_query: K = %d < 1", K);
    MESO_REQUIRE(radius > 0.0f && radius <= 3.0e38f, MESORASI_EINVAL,
                 "mesorasi_ball_query: radius must be finite and > 0");
    MESO_REQUIRE(K <= MESORASI_MAX_K_BALL, MESORASI_EUNSUPPORTED, "mesorasi_ball_query: K = %d > %d", K,
                 MESORASI_MAX_K_BALL);
    if (B == 0 || M == 0) return MESORASI_OK;
    MESO_REQUIRE(N >= 1, MESORASI_EINVAL, "mesorasi_ball_query: N = 0 with M > 0");
    MESO_REQUIRE(xyz && qxyz && nit, MESORASI_EINVAL, "mesorasi_ball_query: NULL xyz, qxyz or nit");
    MESO_REQUIRE(N <= 0x7fffffff - 64 * (kBqChunks + 1) && M <= 0x7fffffff, MESORASI_EUNSUPPORTED, "mesorasi_ball_query: N or M too large");
    const float r2 = radius * radius;
    const int64_t BM = B * M;
    const int64_t blocks = ceil_div(BM, kBqWaves);
    MESO_REQUIRE(blocks <= 0x7fffffff, MESORASI_EUNSUPPORTED, "mesorasi_ball_query: too many queries");
    ball_query_kernel<<<dim3((unsigned)blocks), dim3(64 * kBqWaves), 0, as_stream(stream)>>>(
        xyz, qxyz, BM, (int)N, (int)M, r2, K, nit, cnt);
    return after_launch("mesorasi_ball_query");
}

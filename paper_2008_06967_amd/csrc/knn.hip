// k-nearest-neighbour search and 3-NN interpolation on gfx950.
//
// kNN: the DGCNN neighbor search in the previous module's output space
// (Sec. 4.1 "Work Flow").  A workgroup of 8 waves serves 32 queries of one
// cloud (4 per wave).  Reference points stream through LDS in tiles of 64;
// lane l of every wave computes the distance from reference l of the tile
// to each of its wave's 4 queries (query rows are read from LDS by
// broadcast).  Each query's running top-K lives distributed over the wave:
// lane i holds the i-th smallest (distance, index) pair.  Candidates below
// the current K-th distance are inserted one at a time in index order with a
// ballot (insert position) and a one-lane shift, which reproduces the exact
// (distance, index) order of a stable sort.
//
// interpolate3: feature propagation by inverse squared-distance weights
// over the 3 nearest coarse points (the three_interpolate kernel of the
// PointNet++ segmentation baseline, Sec. 5 "Software Setup").  One thread
// per destination point keeps its 3 nearest in registers while source
// points stream through LDS; the workgroup then interpolates all channels
// with coalesced row reads.
#include "common.h"

namespace meso {

constexpr int kKnnWaves = 8;
constexpr int kKnnQpw = 4;
constexpr int kKnnQpb = kKnnWaves * kKnnQpw;
constexpr int kKnnTile = 64;

__global__ __launch_bounds__(64 * kKnnWaves) void knn_kernel(const float* __restrict__ ref, int64_t ldr,
                                                             const float* __restrict__ query, int64_t ldq, int N, int M,
                                                             int C, int Cs, int K, int qblocks,
                                                             int32_t* __restrict__ nit, float* __restrict__ dist) {
    extern __shared__ float smem[];
    float* sR = smem;                       // [kKnnTile][Cs]   (Cs odd: conflict-free per-lane rows)
    float* sQ = smem + kKnnTile * Cs;       // [kKnnQpb][C]     (read by broadcast)
    const int64_t b = blockIdx.x / qblocks;
    const int q0 = (blockIdx.x % qblocks) * kKnnQpb;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const float inf = __builtin_huge_valf();

    for (int e = tid; e < kKnnQpb * C; e += 64 * kKnnWaves) {
        const int qq = e / C, c = e - qq * C;
        const int qi = q0 + qq;
        sQ[e] = qi < M ? query[(b * M + qi) * ldq + c] : 0.0f;
    }

    float td[kKnnQpw], thr[kKnnQpw];
    int tj[kKnnQpw];
#pragma unroll
    for (int qq = 0; qq < kKnnQpw; ++qq) {
        td[qq] = inf;
        tj[qq] = 0x7fffffff;
        thr[qq] = inf;
    }

    for (int t0 = 0; t0 < N; t0 += kKnnTile) {
        __syncthreads();
        for (int e = tid; e < kKnnTile * C; e += 64 * kKnnWaves) {
            const int r = e / C, c = e - r * C;
            const int j = t0 + r;
            sR[r * Cs + c] = j < N ? ref[(b * N + j) * ldr + c] : 0.0f;
        }
        __syncthreads();
        const int j = t0 + lane;
        const bool valid = j < N;
        float d[kKnnQpw];
#pragma unroll
        for (int qq = 0; qq < kKnnQpw; ++qq) d[qq] = 0.0f;
        const float* rr = sR + lane * Cs;
        const float* qb = sQ + wave * kKnnQpw * C;
        for (int c = 0; c < C; ++c) {
            const float r = rr[c];
#pragma unroll
            for (int qq = 0; qq < kKnnQpw; ++qq) {
                const float t = r - qb[qq * C + c];
                d[qq] = __builtin_fmaf(t, t, d[qq]);
            }
        }
#pragma unroll
        for (int qq = 0; qq < kKnnQpw; ++qq) {
            uint64_t mask = ballot(valid && d[qq] < thr[qq]);
            while (mask) {
                const int l = __builtin_ctzll(mask);
                mask &= mask - 1;
                const float dc = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(d[qq]), l));
                if (dc < thr[qq]) {
                    const int jc = t0 + l;
                    // every stored entry has a smaller index, so it precedes the
                    // candidate iff its distance is <= dc
                    const int pos = __builtin_popcountll(ballot(td[qq] <= dc));
                    const float sd = __shfl_up(td[qq], 1);
                    const int sj = __shfl_up(tj[qq], 1);
                    if (lane == pos) {
                        td[qq] = dc;
                        tj[qq] = jc;
                    } else if (lane > pos) {
                        td[qq] = sd;
                        tj[qq] = sj;
                    }
                    if (lane >= K) {
                        td[qq] = inf;
                        tj[qq] = 0x7fffffff;
                    }
                    thr[qq] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(td[qq]), K - 1));
                }
            }
        }
    }
#pragma unroll
    for (int qq = 0; qq < kKnnQpw; ++qq) {
        const int qi = q0 + wave * kKnnQpw + qq;
        if (qi < M && lane < K) {
            nit[(b * M + qi) * K + lane] = tj[qq];
            if (dist) dist[(b * M + qi) * K + lane] = td[qq];
        }
    }
}

constexpr int kInterpThreads = 256;
constexpr int kInterpChunk = 1024;

__global__ __launch_bounds__(kInterpThreads) void interp3_kernel(const float* __restrict__ xyz_dst,
                                                                 const float* __restrict__ xyz_src,
                                                                 const float* __restrict__ f_src, int64_t lds, int Nd,
                                                                 int Ns, int C, float* __restrict__ f_dst, int64_t ldd,
                                                                 int dblocks) {
    __shared__ float sx[kInterpChunk], sy[kInterpChunk], sz[kInterpChunk];
    __shared__ int s_j[kInterpThreads][3];
    __shared__ float s_w[kInterpThreads][3];
    const int64_t b = blockIdx.x / dblocks;
    const int d0 = (blockIdx.x % dblocks) * kInterpThreads;
    const int tid = threadIdx.x;
    const int i = d0 + tid;
    const bool valid = i < Nd;
    float qx = 0.0f, qy = 0.0f, qz = 0.0f;
    if (valid) {
        qx = xyz_dst[(b * Nd + i) * 3 + 0];
        qy = xyz_dst[(b * Nd + i) * 3 + 1];
        qz = xyz_dst[(b * Nd + i) * 3 + 2];
    }
    const float inf = __builtin_huge_valf();
    float e0 = inf, e1 = inf, e2 = inf;
    int j0 = 0, j1 = 0, j2 = 0;
    for (int c0 = 0; c0 < Ns; c0 += kInterpChunk) {
        __syncthreads();
        const int n = min(kInterpChunk, Ns - c0);
        for (int t = tid; t < n; t += kInterpThreads) {
            const float* s = xyz_src + (b * Ns + c0 + t) * 3;
            sx[t] = s[0];
            sy[t] = s[1];
            sz[t] = s[2];
        }
        __syncthreads();
        for (int t = 0; t < n; ++t) {
            const float d = dist3(sx[t], sy[t], sz[t], qx, qy, qz);
            if (d < e2) {
                const int j = c0 + t;
                if (d < e1) {
                    e2 = e1;
                    j2 = j1;
                    if (d < e0) {
                        e1 = e0;
                        j1 = j0;
                        e0 = d;
                        j0 = j;
                    } else {
                        e1 = d;
                        j1 = j;
                    }
                } else {
                    e2 = d;
                    j2 = j;
                }
            }
        }
    }
    const float w0 = 1.0f / fmaxf(e0, 1e-10f);
    const float w1 = 1.0f / fmaxf(e1, 1e-10f);
    const float w2 = 1.0f / fmaxf(e2, 1e-10f);
    const float ws = w0 + w1 + w2;
    s_j[tid][0] = j0;
    s_j[tid][1] = j1;
    s_j[tid][2] = j2;
    s_w[tid][0] = w0 / ws;
    s_w[tid][1] = w1 / ws;
    s_w[tid][2] = w2 / ws;
    __syncthreads();
    const int nd = min(kInterpThreads, Nd - d0);
    const float* fs = f_src + b * (int64_t)Ns * lds;
    for (int e = tid; e < nd * C; e += kInterpThreads) {
        const int r = e / C, c = e - r * C;
        const float v = s_w[r][0] * fs[(int64_t)s_j[r][0] * lds + c] + s_w[r][1] * fs[(int64_t)s_j[r][1] * lds + c] +
                        s_w[r][2] * fs[(int64_t)s_j[r][2] * lds + c];
        f_dst[(b * Nd + d0 + r) * ldd + c] = v;
    }
}

}  // namespace meso

using namespace meso;

extern "C" int mesorasi_knn(const float* ref, int64_t ld_ref, const float* query, int64_t ld_query, int64_t B,
                            int64_t N, int64_t M, int32_t C, int32_t K, int32_t* nit, float* dist, void* stream) {
    MESO_REQUIRE(B >= 0 && N >= 0 && M >= 0, MESORASI_EINVAL, "mesorasi_knn: negative size");
    MESO_REQUIRE(C >= 1 && K >= 1, MESORASI_EINVAL, "mesorasi_knn: C = %d, K = %d", C, K);
    MESO_REQUIRE(ld_ref >= C && ld_query >= C, MESORASI_EINVAL, "mesorasi_knn: leading dimension < C");
    MESO_REQUIRE(K <= MESORASI_MAX_K_KNN, MESORASI_EUNSUPPORTED, "mesorasi_knn: K = %d > %d", K, MESORASI_MAX_K_KNN);
    MESO_REQUIRE(C <= MESORASI_MAX_C_KNN, MESORASI_EUNSUPPORTED, "mesorasi_knn: C = %d > %d", C, MESORASI_MAX_C_KNN);
    if (B == 0 || M == 0) return MESORASI_OK;
    MESO_REQUIRE(K <= N, MESORASI_EINVAL, "mesorasi_knn: K = %d > N = %lld", K, (long long)N);
    MESO_REQUIRE(ref && query && nit, MESORASI_EINVAL, "mesorasi_knn: NULL ref, query or nit");
    MESO_REQUIRE(N <= 0x7fffffff - 64 && M <= 0x7fffffff, MESORASI_EUNSUPPORTED, "mesorasi_knn: size");
    const int qblocks = (int)ceil_div(M, kKnnQpb);
    const int64_t blocks = B * qblocks;
    MESO_REQUIRE(blocks <= 0x7fffffff, MESORASI_EUNSUPPORTED, "mesorasi_knn: too many queries");
    const int Cs = C | 1;
    const size_t lds = sizeof(float) * ((size_t)kKnnTile * Cs + (size_t)kKnnQpb * C);
    knn_kernel<<<dim3((unsigned)blocks), dim3(64 * kKnnWaves), lds, as_stream(stream)>>>(
        ref, ld_ref, query, ld_query, (int)N, (int)M, C, Cs, K, qblocks, nit, dist);
    return after_launch("mesorasi_knn");
}

extern "C" int mesorasi_interpolate3(const float* xyz_dst, const float* xyz_src, const float* f_src, int64_t ld_src,
                                     int64_t B, int64_t Nd, int64_t Ns, int32_t C, float* f_dst, int64_t ld_dst,
                                     void* stream) {
    MESO_REQUIRE(B >= 0 && Nd >= 0 && Ns >= 0, MESORASI_EINVAL, "mesorasi_interpolate3: negative size");
    MESO_REQUIRE(C >= 1 && ld_src >= C && ld_dst >= C, MESORASI_EINVAL, "mesorasi_interpolate3: C / ld");
    if (B == 0 || Nd == 0) return MESORASI_OK;
    MESO_REQUIRE(Ns >= 3, MESORASI_EINVAL, "mesorasi_interpolate3: Ns = %lld < 3", (long long)Ns);
    MESO_REQUIRE(xyz_dst && xyz_src && f_src && f_dst, MESORASI_EINVAL, "mesorasi_interpolate3: NULL pointer");
    MESO_REQUIRE(Nd <= 0x7fffffff && Ns <= 0x7fffffff, MESORASI_EUNSUPPORTED, "mesorasi_interpolate3: size");
    const int dblocks = (int)ceil_div(Nd, kInterpThreads);
    const int64_t blocks = B * dblocks;
    MESO_REQUIRE(blocks <= 0x7fffffff, MESORASI_EUNSUPPORTED, "mesorasi_interpolate3: too many points");
    interp3_kernel<<<dim3((unsigned)blocks), dim3(kInterpThreads), 0, as_stream(stream)>>>(
        xyz_dst, xyz_src, f_src, ld_src, (int)Nd, (int)Ns, C, f_dst, ld_dst, dblocks);
    return after_launch("mesorasi_interpolate3");
}

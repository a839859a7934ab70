// k-nearest-neighbour search and 3-NN interpolation on gfx950.
//
// kNN: the DGCNN neighbor search in the previous module's output space
// (Sec. 5.1 "Work Flow").  A workgroup of 8 waves serves 32 queries of one
// cloud (4 per wave).  Reference points stream through LDS in tiles of 64;
// lane l of every wave computes the distance from reference l of the tile
// to each of its wave's 4 queries (query rows are read from LDS by
// broadcast).  Each query's running top-K lives distributed over the wave:
// lane i holds the i-th smallest (distance, index) pair.  Candidates below
// the current K-th distance are inserted one at a time in index order with a
// ballot (insert position) and a one-lane shift, which reproduces the exact
// (distance, index) order of a stable sort; a tile with many candidates
// (the first ones) is instead sorted across the wave with a bitonic network
// and merged into the list, in the same (distance, index) order.
//
// interpolate3: feature propagation by inverse squared-distance weights
// over the 3 nearest coarse points (the three_interpolate kernel of the
// PointNet++ segmentation baseline, Sec. 6 "Software Setup"); layout at the
// kernel.
#include "common.h"

namespace meso {

constexpr int kKnnWaves = 8;
constexpr int kKnnQpw = 4;
constexpr int kKnnQpb = kKnnWaves * kKnnQpw;
constexpr int kKnnTile = 64;
constexpr int kKnnSerialMax = 6;   // above this many candidates a tile is sorted and merged

__device__ __forceinline__ bool pair_before(float d, int j, float e, int je) { return d < e || (d == e && j < je); }

// One compare-exchange step across lanes lane and lane ^ jm; `asc` says
// whether this lane's block is sorted ascending.
__device__ __forceinline__ void cx_step(float& d, int& j, int jm, bool asc, int lane) {
    const float od = __shfl_xor(d, jm);
    const int oj = __shfl_xor(j, jm);
    const bool lower = (lane & jm) == 0;
    const bool other_first = pair_before(od, oj, d, j);
    const bool take = (lower == asc) ? other_first : !other_first;
    d = take ? od : d;
    j = take ? oj : j;
}

// Bitonic sort of one (distance, index) pair per lane, ascending over the
// wave in (distance, index) order.
__device__ __forceinline__ void wave_sort_pairs(float& d, int& j, int lane) {
#pragma unroll
    for (int k = 2; k <= 64; k <<= 1)
#pragma unroll
        for (int jm = k >> 1; jm > 0; jm >>= 1) cx_step(d, j, jm, (lane & k) == 0 || k == 64, lane);
}

// (td, tj): an ascending list over the lanes; (sd, sj): another.  Leaves in
// (td, tj) the 64 smallest of both, ascending: the element-wise minimum of
// the first list and the reversed second is bitonic, then half-cleaners.
__device__ __forceinline__ void merge_sorted_pairs(float& td, int& tj, float sd, int sj, int lane) {
    const float rd = __shfl(sd, 63 - lane);
    const int rj = __shfl(sj, 63 - lane);
    if (pair_before(rd, rj, td, tj)) {
        td = rd;
        tj = rj;
    }
#pragma unroll
    for (int jm = 32; jm > 0; jm >>= 1) cx_step(td, tj, jm, true, lane);
}

__global__ __launch_bounds__(64 * kKnnWaves) void knn_kernel(const float* __restrict__ ref, int64_t ldr,
                                                             const float* __restrict__ query, int64_t ldq, int N, int M,
                                                             int C, int Cs, int K, int qblocks, int vec4,
                                                             int32_t* __restrict__ nit, float* __restrict__ dist) {
    extern __shared__ float smem[];
    float* sR = smem;                       // [kKnnTile][Cs]   (per-lane rows; stride odd, or 4 mod 32 for
                                            //  16-byte reads: conflict-free either way)
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
        if (vec4) {
            const int C4 = C >> 2;
            for (int e = tid; e < kKnnTile * C4; e += 64 * kKnnWaves) {
                const int r = e / C4, c = (e - r * C4) << 2;
                const int j = t0 + r;
                const float4 v = j < N ? *reinterpret_cast<const float4*>(ref + (b * N + j) * ldr + c)
                                       : make_float4(0.f, 0.f, 0.f, 0.f);
                *reinterpret_cast<float4*>(sR + r * Cs + c) = v;
            }
        } else {
            for (int e = tid; e < kKnnTile * C; e += 64 * kKnnWaves) {
                const int r = e / C, c = e - r * C;
                const int j = t0 + r;
                sR[r * Cs + c] = j < N ? ref[(b * N + j) * ldr + c] : 0.0f;
            }
        }
        __syncthreads();
        const int j = t0 + lane;
        const bool valid = j < N;
        float d[kKnnQpw];
#pragma unroll
        for (int qq = 0; qq < kKnnQpw; ++qq) d[qq] = 0.0f;
        const float* rr = sR + lane * Cs;
        const float* qb = sQ + wave * kKnnQpw * C;
        if (vec4) {
            // four channels per 16-byte read (the reference row per lane, the
            // query rows by broadcast); the sum stays in channel order
            for (int c = 0; c < C; c += 4) {
                const float4 r = *reinterpret_cast<const float4*>(rr + c);
#pragma unroll
                for (int qq = 0; qq < kKnnQpw; ++qq) {
                    const float4 qv = *reinterpret_cast<const float4*>(qb + qq * C + c);
                    float t = r.x - qv.x;
                    d[qq] = __builtin_fmaf(t, t, d[qq]);
                    t = r.y - qv.y;
                    d[qq] = __builtin_fmaf(t, t, d[qq]);
                    t = r.z - qv.z;
                    d[qq] = __builtin_fmaf(t, t, d[qq]);
                    t = r.w - qv.w;
                    d[qq] = __builtin_fmaf(t, t, d[qq]);
                }
            }
        } else {
            for (int c = 0; c < C; ++c) {
                const float r = rr[c];
#pragma unroll
                for (int qq = 0; qq < kKnnQpw; ++qq) {
                    const float t = r - qb[qq * C + c];
                    d[qq] = __builtin_fmaf(t, t, d[qq]);
                }
            }
        }
#pragma unroll
        for (int qq = 0; qq < kKnnQpw; ++qq) {
            uint64_t mask = ballot(valid && d[qq] < thr[qq]);
            if (__builtin_popcountll(mask) > kKnnSerialMax) {
                // many candidates (the first tiles): sort the tile's (distance,
                // index) pairs across the wave, then merge them into the list
                const bool cand = (mask >> lane) & 1ull;
                float sd = cand ? d[qq] : inf;
                int sj = cand ? t0 + lane : 0x7fffffff;
                wave_sort_pairs(sd, sj, lane);
                merge_sorted_pairs(td[qq], tj[qq], sd, sj, lane);
                if (lane >= K) {
                    td[qq] = inf;
                    tj[qq] = 0x7fffffff;
                }
                thr[qq] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(td[qq]), K - 1));
                mask = 0;
            }
            while (mask) {
                const int l = __builtin_ctzll(mask);
                mask &= mask - 1;
                const float dc = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(d[qq]), l));
                if (dc < thr[qq]) {
                    const int jc = t0 + l;
                    // every stored entry has a smaller index, so it precedes the
                    // candidate iff its distance is <= dc
                    const int pos = __builtin_popcountll(ballot(td[qq] <= dc));
                    // lane i takes lane i-1's entry: one DPP wave_shr:1 each
                    // (lane 0 never uses it)
                    const float sd = __int_as_float(
                        __builtin_amdgcn_update_dpp(0, __float_as_int(td[qq]), 0x138, 0xf, 0xf, false));
                    const int sj = __builtin_amdgcn_update_dpp(0, tj[qq], 0x138, 0xf, 0xf, false);
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

// Register form for clouds of at most 64 * NT points: every wave first
// computes the distances from its 4 queries to all references (reference
// t * 64 + l in lane l, register t), then selects per query:
//  1. tau = the K-th smallest of the 64 lane minima.  These are K distinct
//     references, so tau bounds the K-th smallest distance from above and
//     every reference of the exact top K has d <= tau; for random layouts
//     only a few more than K references do.
//  2. The candidates d <= tau are compacted through LDS (64 at a time),
//     sorted across the wave in (distance, index) order and merged into
//     the list: the same exact order as the streaming form, with one sort
//     and one scan per query instead of a sorted merge or an insert per
//     improving candidate.
template <int NT>
__global__ __launch_bounds__(64 * kKnnWaves) void knn_reg_kernel(const float* __restrict__ ref, int64_t ldr,
                                                                 const float* __restrict__ query, int64_t ldq,
                                                                 int N, int M, int C, int Cs, int K, int qblocks,
                                                                 int vec4, int32_t* __restrict__ nit,
                                                                 float* __restrict__ dist) {
    extern __shared__ float smem[];
    float* sR = smem;                                    // [kKnnTile][Cs]
    float* sQ = smem + kKnnTile * Cs;                    // [kKnnQpb][C]
    float* sCd = sQ + kKnnQpb * C;                       // [kKnnWaves][64] candidate distances
    int* sCj = reinterpret_cast<int*>(sCd + kKnnWaves * 64);   // [kKnnWaves][64] candidate indices
    const int64_t b = blockIdx.x / qblocks;
    const int q0 = (blockIdx.x % qblocks) * kKnnQpb;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const float inf = __builtin_huge_valf();
    const int nt = (N + kKnnTile - 1) / kKnnTile;

    for (int e = tid; e < kKnnQpb * C; e += 64 * kKnnWaves) {
        const int qq = e / C, c = e - qq * C;
        const int qi = q0 + qq;
        sQ[e] = qi < M ? query[(b * M + qi) * ldq + c] : 0.0f;
    }

    // 1. all distances, in the channel order of the oracle
    float d[kKnnQpw][NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
#pragma unroll
        for (int qq = 0; qq < kKnnQpw; ++qq) d[qq][t] = inf;
        if (t < nt) {
            const int t0 = t * kKnnTile;
            __syncthreads();
            if (vec4) {
                const int C4 = C >> 2;
                for (int e = tid; e < kKnnTile * C4; e += 64 * kKnnWaves) {
                    const int r = e / C4, c = (e - r * C4) << 2;
                    const int j = t0 + r;
                    const float4 v = j < N ? *reinterpret_cast<const float4*>(ref + (b * N + j) * ldr + c)
                                           : make_float4(0.f, 0.f, 0.f, 0.f);
                    *reinterpret_cast<float4*>(sR + r * Cs + c) = v;
                }
            } else {
                for (int e = tid; e < kKnnTile * C; e += 64 * kKnnWaves) {
                    const int r = e / C, c = e - r * C;
                    const int j = t0 + r;
                    sR[r * Cs + c] = j < N ? ref[(b * N + j) * ldr + c] : 0.0f;
                }
            }
            __syncthreads();
            float a[kKnnQpw];
#pragma unroll
            for (int qq = 0; qq < kKnnQpw; ++qq) a[qq] = 0.0f;
            const float* rr = sR + lane * Cs;
            const float* qb = sQ + wave * kKnnQpw * C;
            if (vec4) {
                for (int c = 0; c < C; c += 4) {
                    const float4 r = *reinterpret_cast<const float4*>(rr + c);
#pragma unroll
                    for (int qq = 0; qq < kKnnQpw; ++qq) {
                        const float4 qv = *reinterpret_cast<const float4*>(qb + qq * C + c);
                        float u = r.x - qv.x;
                        a[qq] = __builtin_fmaf(u, u, a[qq]);
                        u = r.y - qv.y;
                        a[qq] = __builtin_fmaf(u, u, a[qq]);
                        u = r.z - qv.z;
                        a[qq] = __builtin_fmaf(u, u, a[qq]);
                        u = r.w - qv.w;
                        a[qq] = __builtin_fmaf(u, u, a[qq]);
                    }
                }
            } else {
                for (int c = 0; c < C; ++c) {
                    const float r = rr[c];
#pragma unroll
                    for (int qq = 0; qq < kKnnQpw; ++qq) {
                        const float u = r - qb[qq * C + c];
                        a[qq] = __builtin_fmaf(u, u, a[qq]);
                    }
                }
            }
            const bool valid = t0 + lane < N;
#pragma unroll
            for (int qq = 0; qq < kKnnQpw; ++qq) d[qq][t] = valid ? a[qq] : inf;
        }
    }

    // 2. per query: threshold, candidates, exact order
    float* cd = sCd + wave * 64;
    int* cj = sCj + wave * 64;
#pragma unroll
    for (int qq = 0; qq < kKnnQpw; ++qq) {
        float mn = inf;
#pragma unroll
        for (int t = 0; t < NT; ++t) mn = fminf(mn, d[qq][t]);
        float sv = mn;
        int sl = lane;
        wave_sort_pairs(sv, sl, lane);
        const float tau = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(sv), K - 1));
        // candidates of this lane and their offsets (exclusive scan over lanes)
        int cnt = 0;
#pragma unroll
        for (int t = 0; t < NT; ++t) cnt += (t * kKnnTile + lane < N && d[qq][t] <= tau) ? 1 : 0;
        int incl = cnt;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int v = __shfl_up(incl, o);
            incl += lane >= o ? v : 0;
        }
        const int total = __builtin_amdgcn_readlane(incl, 63);
        const int off = incl - cnt;
        float td = inf;
        int tj = 0x7fffffff;
        for (int base = 0; base < total; base += 64) {
            int o = off;
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                const int j = t * kKnnTile + lane;
                if (j < N && d[qq][t] <= tau) {
                    if (o >= base && o < base + 64) {
                        cd[o - base] = d[qq][t];
                        cj[o - base] = j;
                    }
                    ++o;
                }
            }
            __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
            const bool have = lane < total - base;
            float ed = have ? cd[lane] : inf;
            int ej = have ? cj[lane] : 0x7fffffff;
            __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
            wave_sort_pairs(ed, ej, lane);
            if (base == 0) {
                td = ed;
                tj = ej;
            } else {
                merge_sorted_pairs(td, tj, ed, ej, lane);
            }
        }
        const int qi = q0 + wave * kKnnQpw + qq;
        if (qi < M && lane < K) {
            nit[(b * M + qi) * K + lane] = tj;
            if (dist) dist[(b * M + qi) * K + lane] = td;
        }
    }
}

constexpr int kIpWaves = 4;
constexpr int kIpDests = 128;    // destinations per workgroup, two per lane
constexpr int kIpChunk = 1024;   // sources staged in LDS per pass

// insert (d, j) into an ascending top-3 when sources arrive in index order:
// strict < keeps the earlier index first on equal distances
__device__ __forceinline__ void top3_insert(float d, int j, float (&e)[3], int (&jj)[3]) {
    if (d < e[2]) {
        if (d < e[1]) {
            e[2] = e[1];
            jj[2] = jj[1];
            if (d < e[0]) {
                e[1] = e[0];
                jj[1] = jj[0];
                e[0] = d;
                jj[0] = j;
            } else {
                e[1] = d;
                jj[1] = j;
            }
        } else {
            e[2] = d;
            jj[2] = j;
        }
    }
}

// the same for candidates in any order: (distance, index) lexicographic
__device__ __forceinline__ bool before(float d, int j, float e, int je) { return d < e || (d == e && j < je); }
__device__ __forceinline__ void top3_merge(float d, int j, float (&e)[3], int (&jj)[3]) {
    if (before(d, j, e[2], jj[2])) {
        if (before(d, j, e[1], jj[1])) {
            e[2] = e[1];
            jj[2] = jj[1];
            if (before(d, j, e[0], jj[0])) {
                e[1] = e[0];
                jj[1] = jj[0];
                e[0] = d;
                jj[0] = j;
            } else {
                e[1] = d;
                jj[1] = j;
            }
        } else {
            e[2] = d;
            jj[2] = j;
        }
    }
}

// 3-NN interpolation.  A workgroup serves 128 destinations of one cloud,
// two per lane; its four waves split every staged chunk of sources into
// quarters, each keeping a top-3 per destination over its quarter
// (sources read four at a time with 16-byte LDS broadcasts).  The four
// lists are merged per destination in (distance, index) order, then the
// workgroup interpolates all channels with coalesced row reads.
__global__ __launch_bounds__(64 * kIpWaves) void interp3_kernel(const float* __restrict__ xyz_dst,
                                                                const float* __restrict__ xyz_src,
                                                                const float* __restrict__ f_src, int64_t lds, int Nd,
                                                                int Ns, int C, float* __restrict__ f_dst, int64_t ldd,
                                                                int dblocks, int vec4) {
    __shared__ __attribute__((aligned(16))) float sx[kIpChunk + 16], sy[kIpChunk + 16], sz[kIpChunk + 16];
    __shared__ float s_e[kIpWaves][kIpDests][3];
    __shared__ int s_jj[kIpWaves][kIpDests][3];
    __shared__ int s_j[kIpDests][3];
    __shared__ float s_w[kIpDests][3];
    const int64_t b = blockIdx.x / dblocks;
    const int d0 = (blockIdx.x % dblocks) * kIpDests;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const float inf = __builtin_huge_valf();

    float qx[2], qy[2], qz[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int i = d0 + 64 * h + lane;
        const int ic = i < Nd ? i : Nd - 1;    // a clamped destination computes unused values
        qx[h] = xyz_dst[(b * Nd + ic) * 3 + 0];
        qy[h] = xyz_dst[(b * Nd + ic) * 3 + 1];
        qz[h] = xyz_dst[(b * Nd + ic) * 3 + 2];
    }
    float e[2][3];
    int jj[2][3];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int k = 0; k < 3; ++k) {
            e[h][k] = inf;
            jj[h][k] = 0x7fffffff;
        }

    for (int c0 = 0; c0 < Ns; c0 += kIpChunk) {
        __syncthreads();
        const int n = min(kIpChunk, Ns - c0);
        for (int t = tid; t < n + 16; t += 64 * kIpWaves) {
            float x = inf, y = inf, z = inf;      // padding: infinite distance, never inserted
            if (t < n) {
                const float* src = xyz_src + (b * Ns + c0 + t) * 3;
                x = src[0];
                y = src[1];
                z = src[2];
            }
            sx[t] = x;
            sy[t] = y;
            sz[t] = z;
        }
        __syncthreads();
        const int qn = ((n + 15) / 16) * 4;     // per-wave quarter, a multiple of 4
        const int t_lo = wave * qn;
        for (int t = t_lo; t < t_lo + qn; t += 4) {
            const float4 vx = *reinterpret_cast<const float4*>(&sx[t]);
            const float4 vy = *reinterpret_cast<const float4*>(&sy[t]);
            const float4 vz = *reinterpret_cast<const float4*>(&sz[t]);
            const float ax[4] = {vx.x, vx.y, vx.z, vx.w}, ay[4] = {vy.x, vy.y, vy.z, vy.w},
                        az[4] = {vz.x, vz.y, vz.z, vz.w};
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int j = c0 + t + u;
#pragma unroll
                for (int h = 0; h < 2; ++h) top3_insert(dist3(ax[u], ay[u], az[u], qx[h], qy[h], qz[h]), j, e[h], jj[h]);
            }
        }
    }
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int k = 0; k < 3; ++k) {
            s_e[wave][64 * h + lane][k] = e[h][k];
            s_jj[wave][64 * h + lane][k] = jj[h][k];
        }
    __syncthreads();
    if (tid < kIpDests) {
        float f[3] = {inf, inf, inf};
        int fj[3] = {0x7fffffff, 0x7fffffff, 0x7fffffff};
        for (int w = 0; w < kIpWaves; ++w)
#pragma unroll
            for (int k = 0; k < 3; ++k) top3_merge(s_e[w][tid][k], s_jj[w][tid][k], f, fj);
        const float w0 = 1.0f / fmaxf(f[0], 1e-10f);
        const float w1 = 1.0f / fmaxf(f[1], 1e-10f);
        const float w2 = 1.0f / fmaxf(f[2], 1e-10f);
        const float ws = w0 + w1 + w2;
        s_j[tid][0] = fj[0];
        s_j[tid][1] = fj[1];
        s_j[tid][2] = fj[2];
        s_w[tid][0] = w0 / ws;
        s_w[tid][1] = w1 / ws;
        s_w[tid][2] = w2 / ws;
    }
    __syncthreads();
    const int nd = min(kIpDests, Nd - d0);
    const float* fs = f_src + b * (int64_t)Ns * lds;
    if (vec4) {
        // 16-byte rows: four channels per load and store
        const int C4 = C >> 2;
        for (int el = tid; el < nd * C4; el += 64 * kIpWaves) {
            const int r = el / C4, c = (el - r * C4) << 2;
            const float4 a0 = *reinterpret_cast<const float4*>(fs + (int64_t)s_j[r][0] * lds + c);
            const float4 a1 = *reinterpret_cast<const float4*>(fs + (int64_t)s_j[r][1] * lds + c);
            const float4 a2 = *reinterpret_cast<const float4*>(fs + (int64_t)s_j[r][2] * lds + c);
            const float w0 = s_w[r][0], w1 = s_w[r][1], w2 = s_w[r][2];
            float4 v;
            v.x = w0 * a0.x + w1 * a1.x + w2 * a2.x;
            v.y = w0 * a0.y + w1 * a1.y + w2 * a2.y;
            v.z = w0 * a0.z + w1 * a1.z + w2 * a2.z;
            v.w = w0 * a0.w + w1 * a1.w + w2 * a2.w;
            *reinterpret_cast<float4*>(f_dst + (b * Nd + d0 + r) * ldd + c) = v;
        }
        return;
    }
    for (int el = tid; el < nd * C; el += 64 * kIpWaves) {
        const int r = el / C, c = el - r * C;
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
    // 16-byte path: whole 4-channel groups and 16-byte aligned rows; its LDS
    // row stride C + 4 puts 8 consecutive lanes on distinct bank quads
    const int vec4 = C % 4 == 0 && ld_ref % 4 == 0 && aligned(ref, 16) && C % 32 != 28;
    const int Cs = vec4 ? C + 4 : (C | 1);
    const size_t lds = sizeof(float) * ((size_t)kKnnTile * Cs + (size_t)kKnnQpb * C);
    const dim3 grid((unsigned)blocks), block(64 * kKnnWaves);
    hipStream_t s = as_stream(stream);
    // clouds of at most 1024 points: all distances in registers, then one
    // selection per query; larger clouds stream through the running list
    const size_t lds_reg = lds + sizeof(float) * 2 * 64 * kKnnWaves;
    if (N <= 4 * kKnnTile)
        knn_reg_kernel<4><<<grid, block, lds_reg, s>>>(ref, ld_ref, query, ld_query, (int)N, (int)M, C, Cs, K, qblocks,
                                                       vec4, nit, dist);
    else if (N <= 8 * kKnnTile)
        knn_reg_kernel<8><<<grid, block, lds_reg, s>>>(ref, ld_ref, query, ld_query, (int)N, (int)M, C, Cs, K, qblocks,
                                                       vec4, nit, dist);
    else if (N <= 16 * kKnnTile)
        knn_reg_kernel<16><<<grid, block, lds_reg, s>>>(ref, ld_ref, query, ld_query, (int)N, (int)M, C, Cs, K,
                                                        qblocks, vec4, nit, dist);
    else
        knn_kernel<<<grid, block, lds, s>>>(ref, ld_ref, query, ld_query, (int)N, (int)M, C, Cs, K, qblocks, vec4, nit,
                                            dist);
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
    const int dblocks = (int)ceil_div(Nd, kIpDests);
    const int64_t blocks = B * dblocks;
    MESO_REQUIRE(blocks <= 0x7fffffff, MESORASI_EUNSUPPORTED, "mesorasi_interpolate3: too many points");
    const int vec4 = C % 4 == 0 && ld_src % 4 == 0 && ld_dst % 4 == 0 && aligned(f_src, 16) && aligned(f_dst, 16);
    interp3_kernel<<<dim3((unsigned)blocks), dim3(64 * kIpWaves), 0, as_stream(stream)>>>(
        xyz_dst, xyz_src, f_src, ld_src, (int)Nd, (int)Ns, C, f_dst, ld_dst, dblocks, vec4);
    return after_launch("mesorasi_interpolate3");
}

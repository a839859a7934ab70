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
#include <algorithm>
#include <type_traits>

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

// K-th smallest (K <= 64) of one non-negative float per lane (+inf
// allowed), wave-uniform.  Its bits are fixed from the top: a bit stays 0
// when at least K lanes are <= the largest value with the prefix so far and
// that bit 0 (non-negative floats order like their bit patterns).  One
// ballot per bit, no cross-lane data movement.
__device__ __forceinline__ float wave_kth_smallest(float v, int K) {
    const uint32_t x = __float_as_uint(v);
    uint32_t pre = 0;
#pragma unroll
    for (int bit = 30; bit >= 0; --bit) {
        const uint32_t lim = pre | ((1u << bit) - 1u);
        const int n = __builtin_popcountll(ballot(x <= lim));
        pre = n >= K ? pre : (pre | (1u << bit));
    }
    return __uint_as_float(pre);
}

// Rank of this lane's (d, j) among lanes 0 .. n-1 in (distance, index)
// order (indices distinct): the output slot of a candidate, without a sort.
__device__ __forceinline__ int pair_rank(float d, int j, int n) {
    int r = 0;
    for (int l = 0; l < n; ++l) {
        const float dl = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(d), l));
        const int jl = __builtin_amdgcn_readlane(j, l);
        r += (dl < d || (dl == d && jl < j)) ? 1 : 0;
    }
    return r;
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

    // (thr, thrj): the list's K-th entry, (+inf, INT_MAX) while the list is
    // short, so that a candidate whose distance overflowed to +inf is still
    // admitted then, as by the sequential insertion rule
    float td[kKnnQpw], thr[kKnnQpw];
    int tj[kKnnQpw], thrj[kKnnQpw];
#pragma unroll
    for (int qq = 0; qq < kKnnQpw; ++qq) {
        td[qq] = inf;
        tj[qq] = 0x7fffffff;
        thr[qq] = inf;
        thrj[qq] = 0x7fffffff;
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
            uint64_t mask = ballot(valid && pair_before(d[qq], t0 + lane, thr[qq], thrj[qq]));
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
                thrj[qq] = __builtin_amdgcn_readlane(tj[qq], K - 1);
                mask = 0;
            }
            while (mask) {
                const int l = __builtin_ctzll(mask);
                mask &= mask - 1;
                const float dc = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(d[qq]), l));
                const int jc = t0 + l;
                if (pair_before(dc, jc, thr[qq], thrj[qq])) {
                    // a stored entry has a smaller index than the candidate, so it
                    // precedes it iff its distance is <= dc; an empty slot
                    // (+inf, INT_MAX) never does
                    const int pos = __builtin_popcountll(ballot(pair_before(td[qq], tj[qq], dc, jc)));
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
                    thrj[qq] = __builtin_amdgcn_readlane(tj[qq], K - 1);
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
                                                                 int vec4, int whole, int32_t* __restrict__ nit,
                                                                 float* __restrict__ dist) {
    // whole: the cloud's every reference row is staged once (sR holds NT
    // tiles), instead of one tile per round trip and two barriers
    extern __shared__ float smem[];
    float* sR = smem;                                    // [kKnnTile or NT * kKnnTile][Cs]
    float* sQ = smem + (whole ? NT : 1) * kKnnTile * Cs; // [kKnnQpb][C]
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

    if (whole) {
        for (int e = tid; e < N * C; e += 64 * kKnnWaves) {
            const int r = e / C, c = e - r * C;
            sR[r * Cs + c] = ref[(b * N + r) * ldr + c];
        }
    }

    // 1. all distances, in the channel order of the oracle
    float d[kKnnQpw][NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
#pragma unroll
        for (int qq = 0; qq < kKnnQpw; ++qq) d[qq][t] = inf;
        if (t < nt) {
            const int t0 = t * kKnnTile;
            if (whole) {
                if (t == 0) __syncthreads();
            } else {
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
            }
            float a[kKnnQpw];
#pragma unroll
            for (int qq = 0; qq < kKnnQpw; ++qq) a[qq] = 0.0f;
            // rows past N in the last whole-cloud tile are never staged:
            // their distances are discarded below
            const float* rr = sR + ((whole ? t0 : 0) + lane) * Cs;
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
        const float tau = wave_kth_smallest(mn, K);
        // candidates of this lane and their offsets (exclusive scan over
        // lanes; ballot slots per register would need NT more registers and
        // halve the occupancy)
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
        const int qi = q0 + wave * kKnnQpw + qq;
        if (total <= 64) {
            // the usual case: every candidate's output slot from its rank
            int o = off;
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                const int j = t * kKnnTile + lane;
                if (j < N && d[qq][t] <= tau) {
                    cd[o] = d[qq][t];
                    cj[o] = j;
                    ++o;
                }
            }
            __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
            const bool have = lane < total;
            const float ed = have ? cd[lane] : inf;
            const int ej = have ? cj[lane] : 0x7fffffff;
            __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
            const int rk = pair_rank(ed, ej, total);
            if (have && rk < K && qi < M) {
                nit[(b * M + qi) * K + rk] = ej;
                if (dist) dist[(b * M + qi) * K + rk] = ed;
            }
            continue;
        }
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
        if (qi < M && lane < K) {
            nit[(b * M + qi) * K + lane] = tj;
            if (dist) dist[(b * M + qi) * K + lane] = td;
        }
    }
}

// MFMA form for C in [32, 128] with C % 8 == 0 and N <= 1024 (the DGCNN
// feature-space layers).  The distance a = fl(fl(|x|^2 + |y|^2) - 2 fl(x.y))
// comes from a Gram product on v_mfma_f32_32x32x2_f32; it is only used to
// bound the exact distance d (the fp32 fma chain in channel order):
//   |d - D| <= ((1+u)^2 (1 + gamma_C) - 1) D,   D = |x - y|^2 <= 2(|x|^2 + |y|^2)
//   |a - D| <= (gamma_C + gamma_{C+2} + 3u + O(u^2)) (|x|^2 + |y|^2)
// for any summation order inside the MFMA (products rounded or not), so
// |a - d| <= (4C + 12) u (|x|^2 + |y|^2) to first order; eps below takes
// twice that, plus C * 2^-120 for flushed denormal products, with the
// computed norms.  For C <= 64 the table keeps a rounded to bf16 (a' =
// a(1 + r), |r| <= 2^-8) and the bounds widen by 2^-7 |a'| >= |a' - a|,
// so lower = a' - eps - 2^-7 |a'| <= d <= a' + eps + 2^-7 |a'| = upper
// (fp32 table and no extra term for wider C), and:
//  1. tau = the K-th smallest of the 64 lane minima of upper: K distinct
//     references have d <= tau, so every reference of the exact top K has
//     d <= tau, hence lower <= tau;
//  2. the candidates lower <= tau (or NaN) get their exact d, compacted 64 at a
//     time, and are sorted across the wave in (distance, index) order, as in
//     the register form.  Results are bit-identical to the exact search.
// Workgroup: 32 queries (one MFMA row block), 8 waves.  Phase 1: wave w
// takes reference blocks w, w + 8, ...: its 32 x 32 Gram block from
// registers (query rows fixed, reference rows streamed from global memory,
// the k order of each operand split in two halves like the GEMM), turned
// into a and stored to a 32 x 1032 LDS table: bf16 for C <= 64 (66 KB, so
// two workgroups fit a CU and one's Gram MFMAs overlap the other's
// selection), fp32 above (one workgroup per CU either way, and the bf16
// margin only added candidates).  Phase 2: wave w selects for queries
// 4w .. 4w + 3, reading 4 references per lane per 8- or 16-byte read; its
// candidate list reuses the reference-norm buffer once every wave holds
// its norms in registers.
constexpr int kKnnMfmaLda = 1024 + 8;          // a-table row stride (entries)
constexpr int kKnnMfmaMaxN = 1024;

typedef float knn_f32x16 __attribute__((ext_vector_type(16)));
typedef float knn_f32x4 __attribute__((ext_vector_type(4)));

// Four consecutive table entries as float (bf16 or fp32 table).
__device__ __forceinline__ void load_bounds4(const uint16_t* p, float (&a)[4]) {
    const uint2 v = *reinterpret_cast<const uint2*>(p);
    a[0] = bf16_to_f32(v.x & 0xffffu);
    a[1] = bf16_to_f32(v.x >> 16);
    a[2] = bf16_to_f32(v.y & 0xffffu);
    a[3] = bf16_to_f32(v.y >> 16);
}
__device__ __forceinline__ void load_bounds4(const float* p, float (&a)[4]) {
    const float4 v = *reinterpret_cast<const float4*>(p);
    a[0] = v.x;
    a[1] = v.y;
    a[2] = v.z;
    a[3] = v.w;
}

template <int CH, int QB = kKnnQpb>   // maximum C / 2 (32 or 64); queries per workgroup (32 or 16)
__global__ __launch_bounds__(64 * kKnnWaves) void knn_mfma_kernel(const float* __restrict__ ref, int64_t ldr,
                                                                  const float* __restrict__ query, int64_t ldq,
                                                                  int N, int M, int C, int K, int qblocks,
                                                                  int32_t* __restrict__ nit,
                                                                  float* __restrict__ dist) {
    constexpr bool BF = CH <= 32;                        // bf16 table
    constexpr int QPW = QB / kKnnWaves;                  // queries per wave
    static_assert(QB == 32 || (QB == 16 && !BF), "32 queries, or 16 with the fp32 table");
    using TabT = std::conditional_t<BF, uint16_t, float>;
    extern __shared__ float smem[];
    TabT* sA = reinterpret_cast<TabT*>(smem);            // [32][kKnnMfmaLda] bounds
    const int CQ = C + 4;                                // query row stride: 16-byte lane reads of
                                                         // 32 rows land on distinct bank groups
    float* sQ = smem + QB * kKnnMfmaLda * sizeof(TabT) / sizeof(float);   // [32][CQ]
    float* sNy = sQ + QB * CQ;                      // [1024]
    float* sNx = sNy + kKnnMfmaMaxN;                     // [32]
    uint16_t* sCj = reinterpret_cast<uint16_t*>(sNy);    // [kKnnWaves][4][64], after the norms are read
    const int64_t b = blockIdx.x / qblocks;
    const int q0 = (blockIdx.x % qblocks) * QB;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const float inf = __builtin_huge_valf();
    const int HC = C / 2;

    // 0. queries into LDS, their squared norms
    for (int e = tid; e < QB * C; e += 64 * kKnnWaves) {
        const int qq = e / C, c = e - qq * C;
        const int qi = q0 + qq;
        sQ[qq * CQ + c] = qi < M ? query[(b * M + qi) * ldq + c] : 0.0f;
    }
    __syncthreads();
    if (tid < QB) {
        float nx = 0.0f;
        for (int c = 0; c < C; ++c) nx = __builtin_fmaf(sQ[tid * CQ + c], sQ[tid * CQ + c], nx);
        sNx[tid] = nx;
    }
    const int half = lane >> 5;
    // this lane's query operand: row lane % 32, k half `half` (read from LDS
    // four steps at a time inside the MFMA loop)
    const float* qa = sQ + (lane & 31) * CQ + half * HC;
    __syncthreads();   // sNx visible

    // 1. Gram blocks -> a table; at C <= 64 the next block's reference rows
    //    are loaded while the current block's MFMAs run (two register sets,
    //    pairs of blocks per loop turn so nothing rotates across the loop edge)
    const int nblk = (N + 31) / 32;
    auto load_b = [&](float (&bv)[CH], int blk) {
        const int j = blk * 32 + (lane & 31);
        const float* rr = ref + (b * N + (j < N ? j : N - 1)) * ldr + half * HC;
#pragma unroll
        for (int s4 = 0; s4 < CH / 4; ++s4) {
            const float4 v = s4 * 4 < HC ? *reinterpret_cast<const float4*>(rr + 4 * s4) : make_float4(0.f, 0.f, 0.f, 0.f);
            bv[4 * s4] = v.x; bv[4 * s4 + 1] = v.y; bv[4 * s4 + 2] = v.z; bv[4 * s4 + 3] = v.w;
        }
    };
    auto gram = [&](const float (&bv)[CH], int blk) {
        const int j = blk * 32 + (lane & 31);
        const bool valid = j < N;
        float nyh = 0.0f;
#pragma unroll
        for (int k = 0; k < CH; ++k) nyh = __builtin_fmaf(bv[k], bv[k], nyh);
        const float ny = nyh + __shfl_xor(nyh, 32);
        knn_f32x16 acc;
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[r] = 0.0f;
#pragma unroll
        for (int s4 = 0; s4 < CH / 4; ++s4) {
            const float4 a = s4 * 4 < HC ? *reinterpret_cast<const float4*>(qa + 4 * s4) : make_float4(0.f, 0.f, 0.f, 0.f);
            acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a.x, bv[4 * s4], acc, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a.y, bv[4 * s4 + 1], acc, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a.z, bv[4 * s4 + 2], acc, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a.w, bv[4 * s4 + 3], acc, 0, 0, 0);
        }
        if (lane < 32 && valid) sNy[j] = ny;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int i = 8 * (r >> 2) + 4 * half + (r & 3);
            const float av = valid ? __builtin_fmaf(-2.0f, acc[r], sNx[i] + ny) : inf;
            if constexpr (BF) sA[i * kKnnMfmaLda + j] = f32_to_bf16(av);
            else sA[i * kKnnMfmaLda + j] = av;
        }
    };
    if constexpr (QB == 16) {
        // 16 x 16 blocks on v_mfma_f32_16x16x4_f32: lane l holds reference
        // row 16 blk + l % 16 and query row l % 16 for the channel quarter
        // l / 16 (C % 16 == 0), step s takes channel s of each quarter; the
        // accumulator holds query 4 (l / 16) + r, reference l % 16
        const int QC = C / 4;
        const float* qa4 = sQ + (lane & 15) * CQ + (lane >> 4) * QC;
        const int nblk16 = (N + 15) / 16;
        auto load16 = [&](float (&bv)[CH / 2], int blk) {
            const int j = blk * 16 + (lane & 15);
            const float* rr = ref + (b * N + (j < N ? j : N - 1)) * ldr + (lane >> 4) * QC;
#pragma unroll
            for (int s4 = 0; s4 < CH / 8; ++s4) {
                const float4 v = s4 * 4 < QC ? *reinterpret_cast<const float4*>(rr + 4 * s4) : make_float4(0.f, 0.f, 0.f, 0.f);
                bv[4 * s4] = v.x; bv[4 * s4 + 1] = v.y; bv[4 * s4 + 2] = v.z; bv[4 * s4 + 3] = v.w;
            }
        };
        auto gram16 = [&](const float (&bv)[CH / 2], int blk) {
            const int j = blk * 16 + (lane & 15);
            const bool valid = j < N;
            float nyq = 0.0f;
#pragma unroll
            for (int k = 0; k < CH / 2; ++k) nyq = __builtin_fmaf(bv[k], bv[k], nyq);
            const float ny2 = nyq + __shfl_xor(nyq, 16);
            const float ny = ny2 + __shfl_xor(ny2, 32);
            knn_f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int s4 = 0; s4 < CH / 8; ++s4) {
                const float4 qv = s4 * 4 < QC ? *reinterpret_cast<const float4*>(qa4 + 4 * s4) : make_float4(0.f, 0.f, 0.f, 0.f);
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(qv.x, bv[4 * s4], acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(qv.y, bv[4 * s4 + 1], acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(qv.z, bv[4 * s4 + 2], acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(qv.w, bv[4 * s4 + 3], acc, 0, 0, 0);
            }
            if (lane < 16 && valid) sNy[j] = ny;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int i = 4 * (lane >> 4) + r;
                sA[i * kKnnMfmaLda + j] = valid ? __builtin_fmaf(-2.0f, acc[r], sNx[i] + ny) : inf;
            }
        };
        // the next block's reference rows load while this block's MFMAs run
        // (two register sets, pairs of blocks per loop turn)
        float b0[CH / 2], b1[CH / 2];
        if (wave < nblk16) load16(b0, wave);
        for (int blk = wave; blk < nblk16; blk += 2 * kKnnWaves) {
            const int nb1 = blk + kKnnWaves;
            if (nb1 < nblk16) load16(b1, nb1);
            gram16(b0, blk);
            if (nb1 >= nblk16) break;
            if (nb1 + kKnnWaves < nblk16) load16(b0, nb1 + kKnnWaves);
            gram16(b1, nb1);
        }
    } else if constexpr (CH <= 32) {
        float b0[CH], b1[CH];
        if (wave < nblk) load_b(b0, wave);
        for (int blk = wave; blk < nblk; blk += 2 * kKnnWaves) {
            const int nb1 = blk + kKnnWaves;
            if (nb1 < nblk) load_b(b1, nb1);
            gram(b0, blk);
            if (nb1 >= nblk) break;
            if (nb1 + kKnnWaves < nblk) load_b(b0, nb1 + kKnnWaves);
            gram(b1, nb1);
        }
    } else {
        // 64 words per operand half: one register set (two measured slower)
        float b0[CH];
        for (int blk = wave; blk < nblk; blk += kKnnWaves) {
            load_b(b0, blk);
            gram(b0, blk);
        }
    }
    __syncthreads();

    // 2. selection: for each of the wave's 4 queries a threshold and the
    //    candidate slots (one ballot per register); then the exact distances
    //    of all 4 queries' candidates together (4 independent chains per
    //    lane), then each candidate's output slot from its rank.  A query
    //    with more than 64 candidates is sorted and merged 64 at a time.
    const float kappa = (float)(8 * C + 32) * 0x1p-24f;
    const float tiny = (float)C * 0x1p-120f;
    float nyv[16];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        const float4 v = *reinterpret_cast<const float4*>(sNy + 256 * t + 4 * lane);
        nyv[4 * t] = v.x; nyv[4 * t + 1] = v.y; nyv[4 * t + 2] = v.z; nyv[4 * t + 3] = v.w;
    }
    __syncthreads();   // every wave holds its norms: sNy becomes the candidate lists
    uint16_t* cjw = sCj + wave * (QPW * 64);   // [4][64] candidate indices of this wave
    int total[QPW];
    float tau[QPW];
#pragma unroll
    for (int qq = 0; qq < QPW; ++qq) {
        const int i = wave * QPW + qq;
        const float nxq = sNx[i];
        float lo[16];
        float mn = inf;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            float av4[4];
            load_bounds4(sA + i * kKnnMfmaLda + 256 * t + 4 * lane, av4);
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const bool valid = 256 * t + 4 * lane + u < N;
                const float e = __builtin_fmaf(kappa, nxq + nyv[4 * t + u], tiny) + (BF ? 0x1p-7f * fabsf(av4[u]) : 0.0f);
                const float up = valid ? av4[u] + e : inf;
                lo[4 * t + u] = av4[u] - e;
                mn = fminf(mn, up);
            }
        }
        tau[qq] = wave_kth_smallest(mn, K);
        int tot = 0;
        int slot[16];
#pragma unroll
        for (int t = 0; t < 16; ++t) {
            const int j = 256 * (t >> 2) + 4 * lane + (t & 3);
            const bool c = j < N && !(lo[t] > tau[qq]);   // NaN bounds are candidates
            const uint64_t m = ballot(c);
            slot[t] = c ? tot + mask_rank(m) : -1;
            tot += __builtin_popcountll(m);
        }
        total[qq] = tot;
        if (tot <= 64) {
#pragma unroll
            for (int t = 0; t < 16; ++t)
                if (slot[t] >= 0) cjw[qq * 64 + slot[t]] = (uint16_t)(256 * (t >> 2) + 4 * lane + (t & 3));
        }
    }
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    // exact distances (the oracle's channel order) of this lane's candidate
    // of each query
    int jc[QPW];
    float dx[QPW];
#pragma unroll
    for (int qq = 0; qq < QPW; ++qq) {
        jc[qq] = (total[qq] <= 64 && lane < total[qq]) ? cjw[qq * 64 + lane] : 0;
        dx[qq] = 0.0f;
    }
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    {
        const float* rr[QPW];
        const float* qr[QPW];
#pragma unroll
        for (int qq = 0; qq < QPW; ++qq) {
            rr[qq] = ref + (b * N + jc[qq]) * ldr;
            qr[qq] = sQ + (wave * QPW + qq) * CQ;
        }
#pragma unroll
        for (int c4 = 0; c4 < CH / 2; ++c4) {
            if (c4 * 4 < C) {
#pragma unroll
                for (int qq = 0; qq < QPW; ++qq) {
                    const float4 r = *reinterpret_cast<const float4*>(rr[qq] + 4 * c4);
                    const float4 qv = *reinterpret_cast<const float4*>(qr[qq] + 4 * c4);
                    float u = r.x - qv.x;
                    dx[qq] = __builtin_fmaf(u, u, dx[qq]);
                    u = r.y - qv.y;
                    dx[qq] = __builtin_fmaf(u, u, dx[qq]);
                    u = r.z - qv.z;
                    dx[qq] = __builtin_fmaf(u, u, dx[qq]);
                    u = r.w - qv.w;
                    dx[qq] = __builtin_fmaf(u, u, dx[qq]);
                }
            }
        }
    }
    for (int qq = 0; qq < QPW; ++qq) {
        const int i = wave * QPW + qq;
        const int qi = q0 + i;
        const int tot = total[qq];
        if (tot <= 64) {
            const bool have = lane < tot;
            const float ed = have ? dx[qq] : inf;
            const int ej = have ? jc[qq] : 0x7fffffff;
            const int rk = pair_rank(ed, ej, tot);
            if (have && rk < K && qi < M) {
                nit[(b * M + qi) * K + rk] = ej;
                if (dist) dist[(b * M + qi) * K + rk] = ed;
            }
            continue;
        }
        // many candidates (near-equal distances under wide margins): recompute
        // this query's bounds and take the candidates 64 at a time
        const float nxq = sNx[i];
        int slot[16];
        int t2 = 0;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            float av4[4];
            load_bounds4(sA + i * kKnnMfmaLda + 256 * t + 4 * lane, av4);
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int j = 256 * t + 4 * lane + u;
                const float e = __builtin_fmaf(kappa, nxq + nyv[4 * t + u], tiny) + (BF ? 0x1p-7f * fabsf(av4[u]) : 0.0f);
                const bool c = j < N && !(av4[u] - e > tau[qq]);
                const uint64_t m = ballot(c);
                slot[4 * t + u] = c ? t2 + mask_rank(m) : -1;
                t2 += __builtin_popcountll(m);
            }
        }
        uint16_t* cj = cjw + qq * 64;
        const float* qrow = sQ + i * CQ;
        float td = inf;
        int tj = 0x7fffffff;
        for (int base = 0; base < tot; base += 64) {
#pragma unroll
            for (int t = 0; t < 16; ++t)
                if (slot[t] >= base && slot[t] < base + 64)
                    cj[slot[t] - base] = (uint16_t)(256 * (t >> 2) + 4 * lane + (t & 3));
            __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
            const bool have = lane < tot - base;
            const int jj = have ? cj[lane] : 0;
            __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
            const float* rr = ref + (b * N + jj) * ldr;
            float d = 0.0f;
            for (int c4 = 0; c4 < C / 4; ++c4) {
                const float4 r = *reinterpret_cast<const float4*>(rr + 4 * c4);
                const float4 qv = *reinterpret_cast<const float4*>(qrow + 4 * c4);
                float u = r.x - qv.x;
                d = __builtin_fmaf(u, u, d);
                u = r.y - qv.y;
                d = __builtin_fmaf(u, u, d);
                u = r.z - qv.z;
                d = __builtin_fmaf(u, u, d);
                u = r.w - qv.w;
                d = __builtin_fmaf(u, u, d);
            }
            float ed = have ? d : inf;
            int ej = have ? jj : 0x7fffffff;
            wave_sort_pairs(ed, ej, lane);
            if (base == 0) {
                td = ed;
                tj = ej;
            } else {
                merge_sorted_pairs(td, tj, ed, ej, lane);
            }
        }
        if (qi < M && lane < K) {
            nit[(b * M + qi) * K + lane] = tj;
            if (dist) dist[(b * M + qi) * K + lane] = td;
        }
    }
}

constexpr int kIpWaves = 4;
constexpr int kIpDests = 128;    // destinations per workgroup, two per lane
constexpr int kIpChunk = 1024;   // sources staged in LDS per pass

// insert (d, j) into an ascending top-3 in (distance, index) order (the
// merge of the waves' lists).  An empty slot (+inf, INT_MAX) takes any
// entry, also one whose distance overflowed to +inf.
__device__ __forceinline__ void top3_insert(float d, int j, float (&e)[3], int (&jj)[3]) {
    if (pair_before(d, j, e[2], jj[2])) {
        if (pair_before(d, j, e[1], jj[1])) {
            e[2] = e[1];
            jj[2] = jj[1];
            if (pair_before(d, j, e[0], jj[0])) {
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

// The scan's top-3 of one destination, as distance bits: sources arrive in
// ascending index order, so a source enters only with a strictly smaller
// distance (an equal one has the larger index) and one unsigned compare of
// the bits (distances are >= +0) is the (distance, index) order.  An empty
// slot holds kTopOpen, above the bits of every distance, +inf included (so
// it takes any source, also one whose distance overflowed), and below
// those of the NaN that padding sources carry (never inserted).
constexpr unsigned kTopOpen = 0x7f800001u;

__device__ __forceinline__ void top3_scan_insert(unsigned db, int j, unsigned (&eb)[3], int (&jj)[3]) {
    if (db < eb[2]) {
        const bool b0 = db < eb[0], b1 = db < eb[1];
        const unsigned e0 = eb[0], e1 = eb[1];
        const int j0 = jj[0], j1 = jj[1];
        eb[2] = b1 ? e1 : db;
        jj[2] = b1 ? j1 : j;
        eb[1] = b0 ? e0 : (b1 ? db : e1);
        jj[1] = b0 ? j0 : (b1 ? j : j1);
        eb[0] = b0 ? db : e0;
        jj[0] = b0 ? j : j0;
    }
}

// 3-NN interpolation.  A workgroup serves 128 destinations of one cloud,
// two per lane; its four waves split every staged chunk of sources into
// quarters, each keeping a top-3 per destination over its quarter
// (sources read four at a time with 16-byte LDS broadcasts).  The four
// lists are merged per destination in (distance, index) order, then the
// workgroup interpolates all channels with coalesced row reads.
// SEARCH_ONLY: stop after the merge and write the three indices and squared
// distances (nit, dist [B, Nd, 3]) instead of interpolating.
template <bool SEARCH_ONLY>
__global__ __launch_bounds__(64 * kIpWaves) void interp3_kernel(const float* __restrict__ xyz_dst,
                                                                const float* __restrict__ xyz_src,
                                                                const float* __restrict__ f_src, int64_t lds, int Nd,
                                                                int Ns, int C, float* __restrict__ f_dst, int64_t ldd,
                                                                int dblocks, int vec4, int32_t* __restrict__ nn_out,
                                                                float* __restrict__ d_out) {
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
    unsigned eb[2][3];
    int jj[2][3];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int k = 0; k < 3; ++k) {
            eb[h][k] = kTopOpen;
            jj[h][k] = 0x7fffffff;
        }

    for (int c0 = 0; c0 < Ns; c0 += kIpChunk) {
        __syncthreads();
        const int n = min(kIpChunk, Ns - c0);
        for (int t = tid; t < n + 16; t += 64 * kIpWaves) {
            // padding: NaN coordinates, so a NaN distance that never enters
            float x = __builtin_nanf(""), y = x, z = x;
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
                for (int h = 0; h < 2; ++h)
                    top3_scan_insert(__float_as_uint(dist3(ax[u], ay[u], az[u], qx[h], qy[h], qz[h])), j, eb[h],
                                     jj[h]);
            }
        }
    }
    // back to (distance, index) pairs, an empty slot as (+inf, INT_MAX)
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int k = 0; k < 3; ++k) {
            s_e[wave][64 * h + lane][k] = eb[h][k] == kTopOpen ? inf : __uint_as_float(eb[h][k]);
            s_jj[wave][64 * h + lane][k] = jj[h][k];
        }
    __syncthreads();
    if (tid < kIpDests) {
        float f[3] = {inf, inf, inf};
        int fj[3] = {0x7fffffff, 0x7fffffff, 0x7fffffff};
        for (int w = 0; w < kIpWaves; ++w)
#pragma unroll
            for (int k = 0; k < 3; ++k) top3_insert(s_e[w][tid][k], s_jj[w][tid][k], f, fj);
        if constexpr (SEARCH_ONLY) {
            const int i = d0 + tid;
            if (i < Nd) {
#pragma unroll
                for (int k = 0; k < 3; ++k) {
                    nn_out[(b * Nd + i) * 3 + k] = min(fj[k], Ns - 1);
                    d_out[(b * Nd + i) * 3 + k] = f[k];
                }
            }
        } else {
            const float w0 = 1.0f / fmaxf(f[0], 1e-10f);
            const float w1 = 1.0f / fmaxf(f[1], 1e-10f);
            const float w2 = 1.0f / fmaxf(f[2], 1e-10f);
            const float ws = w0 + w1 + w2;
            // with Ns >= 3 every slot holds a source (any source precedes an
            // empty slot); the min only keeps the row reads below inside f_src
            s_j[tid][0] = min(fj[0], Ns - 1);
            s_j[tid][1] = min(fj[1], Ns - 1);
            s_j[tid][2] = min(fj[2], Ns - 1);
            s_w[tid][0] = w0 / ws;
            s_w[tid][1] = w1 / ws;
            s_w[tid][2] = w2 / ws;
        }
    }
    if constexpr (SEARCH_ONLY) return;
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

// Interpolation from precomputed neighbours: thread e of the grid-stride
// loop takes destination e / C4 and four channels (or one channel without
// 16-byte rows).  The weights are those of interp3_kernel, in the same fp32
// operations, so the two paths agree bit for bit.  ADD: f_dst =
// phi(interpolation + add), phi = ReLU when relu is set (add may be f_dst
// itself: every element is read before the same thread writes it).
template <bool VEC4, bool ADD = false>
__global__ __launch_bounds__(256) void interp3_apply_kernel(const int32_t* __restrict__ nn, const float* __restrict__ dd,
                                                            const float* __restrict__ f_src, int64_t lds, int64_t Nd,
                                                            int Ns, int C, int64_t total, float* f_dst, int64_t ldd,
                                                            const float* add = nullptr, int64_t lda = 0,
                                                            int relu = 0) {
    const int cw = VEC4 ? C >> 2 : C;
    // workgroups are dealt to the 8 XCDs round-robin by id (the grid is a
    // multiple of 8): renumber them so each XCD runs one contiguous range of
    // destinations -- whole clouds -- and gathers its source rows into its
    // own L2 only
    const int64_t lb = (int64_t)(blockIdx.x & 7) * (gridDim.x >> 3) + (blockIdx.x >> 3);
    for (int64_t e = lb * blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t r = e / cw;                // global destination b * Nd + i
        const int c = (int)(e - r * cw) * (VEC4 ? 4 : 1);
        const int64_t b = r / Nd;
        const float w0 = 1.0f / fmaxf(dd[r * 3 + 0], 1e-10f);
        const float w1 = 1.0f / fmaxf(dd[r * 3 + 1], 1e-10f);
        const float w2 = 1.0f / fmaxf(dd[r * 3 + 2], 1e-10f);
        const float ws = w0 + w1 + w2;
        const float u0 = w0 / ws, u1 = w1 / ws, u2 = w2 / ws;
        const float* fs = f_src + b * (int64_t)Ns * lds;
        const float* a0 = fs + (int64_t)nn[r * 3 + 0] * lds + c;
        const float* a1 = fs + (int64_t)nn[r * 3 + 1] * lds + c;
        const float* a2 = fs + (int64_t)nn[r * 3 + 2] * lds + c;
        float* o = f_dst + r * ldd + c;
        if constexpr (VEC4) {
            const float4 x0 = *reinterpret_cast<const float4*>(a0);
            const float4 x1 = *reinterpret_cast<const float4*>(a1);
            const float4 x2 = *reinterpret_cast<const float4*>(a2);
            float4 v;
            v.x = u0 * x0.x + u1 * x1.x + u2 * x2.x;
            v.y = u0 * x0.y + u1 * x1.y + u2 * x2.y;
            v.z = u0 * x0.z + u1 * x1.z + u2 * x2.z;
            v.w = u0 * x0.w + u1 * x1.w + u2 * x2.w;
            if constexpr (ADD) {
                const float4 p = *reinterpret_cast<const float4*>(add + r * lda + c);
                v.x += p.x;
                v.y += p.y;
                v.z += p.z;
                v.w += p.w;
                if (relu) {
                    v.x = v.x > 0.0f ? v.x : 0.0f;
                    v.y = v.y > 0.0f ? v.y : 0.0f;
                    v.z = v.z > 0.0f ? v.z : 0.0f;
                    v.w = v.w > 0.0f ? v.w : 0.0f;
                }
            }
            *reinterpret_cast<float4*>(o) = v;
        } else {
            float v = u0 * *a0 + u1 * *a1 + u2 * *a2;
            if constexpr (ADD) {
                v += add[r * lda + c];
                if (relu) v = v > 0.0f ? v : 0.0f;
            }
            *o = v;
        }
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
    const bool mfma = N <= kKnnMfmaMaxN && C >= 32 && C % 8 == 0 && ld_ref % 4 == 0 && aligned(ref, 16);
    if (mfma) {
        // bounds table (bf16 for C <= 64), query rows, reference norms
        // (later the candidate lists), query norms: 79 KB at C = 64, so two
        // workgroups per CU
        const size_t lds_m = (C <= 64 ? sizeof(uint16_t) : sizeof(float)) * (size_t)kKnnQpb * kKnnMfmaLda +
                             sizeof(float) * ((size_t)kKnnQpb * (C + 4) + kKnnMfmaMaxN + kKnnQpb);
        if (C <= 64) {
            static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(&knn_mfma_kernel<32>),
                                                               hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
            MESO_REQUIRE(attr == hipSuccess, MESORASI_EHIP, "mesorasi_knn: LDS size attribute: %s", hipGetErrorString(attr));
            knn_mfma_kernel<32><<<grid, block, lds_m, s>>>(ref, ld_ref, query, ld_query, (int)N, (int)M, C, K, qblocks,
                                                           nit, dist);
        } else if (C % 16 == 0) {
            // 16 queries per workgroup (fp32 table of 66 KB): two workgroups
            // per CU, so one's Gram MFMAs overlap the other's selection
            constexpr int QB16 = 16;
            const int qb16 = (int)ceil_div(M, QB16);
            MESO_REQUIRE(B * qb16 <= 0x7fffffff, MESORASI_EUNSUPPORTED, "mesorasi_knn: too many queries");
            const size_t lds16 = sizeof(float) * ((size_t)QB16 * kKnnMfmaLda + (size_t)QB16 * (C + 4) + kKnnMfmaMaxN + QB16);
            static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(&knn_mfma_kernel<64, QB16>),
                                                               hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
            MESO_REQUIRE(attr == hipSuccess, MESORASI_EHIP, "mesorasi_knn: LDS size attribute: %s", hipGetErrorString(attr));
            knn_mfma_kernel<64, QB16><<<dim3((unsigned)(B * qb16)), block, lds16, s>>>(ref, ld_ref, query, ld_query, (int)N,
                                                                                    (int)M, C, K, qb16, nit, dist);
        } else {
            static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(&knn_mfma_kernel<64>),
                                                               hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
            MESO_REQUIRE(attr == hipSuccess, MESORASI_EHIP, "mesorasi_knn: LDS size attribute: %s", hipGetErrorString(attr));
            knn_mfma_kernel<64><<<grid, block, lds_m, s>>>(ref, ld_ref, query, ld_query, (int)N, (int)M, C, K, qblocks,
                                                           nit, dist);
        }
    } else if (N <= 16 * kKnnTile) {
        // a cloud of at most 32 KB is staged whole (one round trip instead of
        // one per 64-row tile)
        const int nt_k = N <= 4 * kKnnTile ? 4 : N <= 8 * kKnnTile ? 8 : 16;
        const size_t whole_rows = sizeof(float) * (size_t)nt_k * kKnnTile * Cs;
        const int whole = whole_rows <= 32 * 1024 ? 1 : 0;
        const size_t l = lds_reg + (whole ? whole_rows - sizeof(float) * (size_t)kKnnTile * Cs : 0);
        if (nt_k == 4)
            knn_reg_kernel<4><<<grid, block, l, s>>>(ref, ld_ref, query, ld_query, (int)N, (int)M, C, Cs, K, qblocks,
                                                     vec4, whole, nit, dist);
        else if (nt_k == 8)
            knn_reg_kernel<8><<<grid, block, l, s>>>(ref, ld_ref, query, ld_query, (int)N, (int)M, C, Cs, K, qblocks,
                                                     vec4, whole, nit, dist);
        else
            knn_reg_kernel<16><<<grid, block, l, s>>>(ref, ld_ref, query, ld_query, (int)N, (int)M, C, Cs, K, qblocks,
                                                      vec4, whole, nit, dist);
    } else
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
    interp3_kernel<false><<<dim3((unsigned)blocks), dim3(64 * kIpWaves), 0, as_stream(stream)>>>(
        xyz_dst, xyz_src, f_src, ld_src, (int)Nd, (int)Ns, C, f_dst, ld_dst, dblocks, vec4, nullptr, nullptr);
    return after_launch("mesorasi_interpolate3");
}

extern "C" int mesorasi_three_nn(const float* xyz_dst, const float* xyz_src, int64_t B, int64_t Nd, int64_t Ns,
                                 int32_t* nit, float* dist, void* stream) {
    MESO_REQUIRE(B >= 0 && Nd >= 0 && Ns >= 0, MESORASI_EINVAL, "mesorasi_three_nn: negative size");
    if (B == 0 || Nd == 0) return MESORASI_OK;
    MESO_REQUIRE(Ns >= 3, MESORASI_EINVAL, "mesorasi_three_nn: Ns = %lld < 3", (long long)Ns);
    MESO_REQUIRE(xyz_dst && xyz_src && nit && dist, MESORASI_EINVAL, "mesorasi_three_nn: NULL pointer");
    MESO_REQUIRE(Nd <= 0x7fffffff && Ns <= 0x7fffffff, MESORASI_EUNSUPPORTED, "mesorasi_three_nn: size");
    const int dblocks = (int)ceil_div(Nd, kIpDests);
    const int64_t blocks = B * dblocks;
    MESO_REQUIRE(blocks <= 0x7fffffff, MESORASI_EUNSUPPORTED, "mesorasi_three_nn: too many points");
    interp3_kernel<true><<<dim3((unsigned)blocks), dim3(64 * kIpWaves), 0, as_stream(stream)>>>(
        xyz_dst, xyz_src, nullptr, 0, (int)Nd, (int)Ns, 1, nullptr, 0, dblocks, 0, nit, dist);
    return after_launch("mesorasi_three_nn");
}

extern "C" int mesorasi_interpolate3_apply(const int32_t* nit, const float* dist, const float* f_src, int64_t ld_src,
                                           int64_t B, int64_t Nd, int64_t Ns, int32_t C, float* f_dst, int64_t ld_dst,
                                           void* stream) {
    MESO_REQUIRE(B >= 0 && Nd >= 0 && Ns >= 0, MESORASI_EINVAL, "mesorasi_interpolate3_apply: negative size");
    MESO_REQUIRE(C >= 1 && ld_src >= C && ld_dst >= C, MESORASI_EINVAL, "mesorasi_interpolate3_apply: C / ld");
    if (B == 0 || Nd == 0) return MESORASI_OK;
    MESO_REQUIRE(Ns >= 1, MESORASI_EINVAL, "mesorasi_interpolate3_apply: Ns = 0");
    MESO_REQUIRE(nit && dist && f_src && f_dst, MESORASI_EINVAL, "mesorasi_interpolate3_apply: NULL pointer");
    MESO_REQUIRE(Ns <= 0x7fffffff, MESORASI_EUNSUPPORTED, "mesorasi_interpolate3_apply: size");
    const bool vec4 = C % 4 == 0 && ld_src % 4 == 0 && ld_dst % 4 == 0 && aligned(f_src, 16) && aligned(f_dst, 16);
    const int64_t total = B * Nd * (vec4 ? C / 4 : C);
    const dim3 grid((unsigned)(8 * ceil_div(std::min<int64_t>(ceil_div(total, 256), 8192), 8))), block(256);
    if (vec4)
        interp3_apply_kernel<true><<<grid, block, 0, as_stream(stream)>>>(nit, dist, f_src, ld_src, Nd, (int)Ns, C,
                                                                         total, f_dst, ld_dst);
    else
        interp3_apply_kernel<false><<<grid, block, 0, as_stream(stream)>>>(nit, dist, f_src, ld_src, Nd, (int)Ns, C,
                                                                          total, f_dst, ld_dst);
    return after_launch("mesorasi_interpolate3_apply");
}

extern "C" int mesorasi_interpolate3_add(const int32_t* nit, const float* dist, const float* f_src, int64_t ld_src,
                                         int64_t B, int64_t Nd, int64_t Ns, int32_t C, const float* add,
                                         int64_t ld_add, int32_t relu, float* f_dst, int64_t ld_dst, void* stream) {
    MESO_REQUIRE(B >= 0 && Nd >= 0 && Ns >= 0, MESORASI_EINVAL, "mesorasi_interpolate3_add: negative size");
    MESO_REQUIRE(C >= 1 && ld_src >= C && ld_dst >= C && ld_add >= C, MESORASI_EINVAL,
                 "mesorasi_interpolate3_add: C / ld");
    if (B == 0 || Nd == 0) return MESORASI_OK;
    MESO_REQUIRE(Ns >= 1, MESORASI_EINVAL, "mesorasi_interpolate3_add: Ns = 0");
    MESO_REQUIRE(nit && dist && f_src && add && f_dst, MESORASI_EINVAL, "mesorasi_interpolate3_add: NULL pointer");
    MESO_REQUIRE(add != f_dst || ld_add == ld_dst, MESORASI_EINVAL,
                 "mesorasi_interpolate3_add: add aliases f_dst with another leading dimension");
    MESO_REQUIRE(Ns <= 0x7fffffff, MESORASI_EUNSUPPORTED, "mesorasi_interpolate3_add: size");
    const bool vec4 = C % 4 == 0 && ld_src % 4 == 0 && ld_dst % 4 == 0 && ld_add % 4 == 0 && aligned(f_src, 16) &&
                      aligned(f_dst, 16) && aligned(add, 16);
    const int64_t total = B * Nd * (vec4 ? C / 4 : C);
    const dim3 grid((unsigned)(8 * ceil_div(std::min<int64_t>(ceil_div(total, 256), 8192), 8))), block(256);
    if (vec4)
        interp3_apply_kernel<true, true><<<grid, block, 0, as_stream(stream)>>>(
            nit, dist, f_src, ld_src, Nd, (int)Ns, C, total, f_dst, ld_dst, add, ld_add, relu);
    else
        interp3_apply_kernel<false, true><<<grid, block, 0, as_stream(stream)>>>(
            nit, dist, f_src, ld_src, Nd, (int)Ns, C, total, f_dst, ld_dst, add, ld_add, relu);
    return after_launch("mesorasi_interpolate3_add");
}

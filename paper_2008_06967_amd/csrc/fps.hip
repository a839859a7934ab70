// Farthest-point sampling on gfx950: one workgroup per cloud.
//
// The sampling step of the PointNet++ modules (Sec. 6, "Software Setup")
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
// An iteration: each thread updates its P running minima (as float bits:
// every value is >= 0 or the -1 padding sentinel, so a signed-int min is
// the strict-less minimum in one instruction) and keeps their max and the
// lowest slot holding it (found while the wave max is reduced); a
// fused-DPP butterfly gives the wave max, one ballot the lowest lane
// holding it, and that lane's slot is read out, both wave-uniform, so the
// winner's coordinates are read once with a uniform register index --
// per-lane work after the reduction does not grow with P.  One barrier per
// iteration: the per-wave winners go to a ring of 128
// LDS slot rows indexed by iteration, so a wave that runs ahead writes the
// next row while slower waves still read this one.  The ring also keeps
// the results: every 64 iterations each lane of wave 0 finds the winner of
// one past iteration again from its row (highest distance, lowest wave)
// and stores it, so no wave spends instructions recording the winner on
// the path to the next barrier (doing it per iteration cost about 10 % at
// 8 waves).  A single-wave workgroup needs no barrier at all and keeps its
// results in registers.  The iteration is bound by VALU issue for large P
// (four waves per SIMD at 16 points per thread) and by the reduction chain
// for small P.
//
// From 513 to 8192 points fps_lds_kernel keeps a copy of the coordinates
// in LDS as well, so the winners are exchanged as (distance, index) and the
// new centroid is read from LDS after the block reduction; from 8193 to
// 16384 points fps_skip_kernel orders the cloud spatially and skips the
// updates that provably change nothing; above 32768 points fps_multi_kernel
// spreads a cloud over several workgroups.
#include <algorithm>

#include "common.h"

namespace meso {

template <int T, int P, bool REG_XYZ>
__global__ __launch_bounds__(T) void fps_kernel(const float* __restrict__ xyz, int N, int M, int32_t* __restrict__ idx,
                                                float* __restrict__ cxyz) {
    constexpr int W = T / 64;
    constexpr int R = W > 1 ? 128 : 1;   // ring rows (two result blocks of 64 iterations)
    // per-wave winner of iteration m in row m % R: {dist bits, index, x, y} and z
    __shared__ int4 s_slot[R][W];
    __shared__ float s_z[R][W];

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
    const float x0 = cx, y0 = cy, z0 = cz;
    // Multi-wave: lane l of wave 0 resolves iteration (m_last & ~63) + l
    // from the ring and stores it (iteration 0 is point 0).
    auto resolve = [&](int m_last) {
        const int mi = (m_last & ~63) + lane;
        const int row = mi & (R - 1);
        int best = s_slot[row][0].x, bw = 0;
#pragma unroll
        for (int w = 1; w < W; ++w) {
            const int d = s_slot[row][w].x;
            bw = d > best ? w : bw;
            best = d > best ? d : best;
        }
        const int4 sl = s_slot[row][bw];
        const float sz = s_z[row][bw];
        if (mi <= m_last) {
            const bool first = mi == 0;
            out_idx[mi] = first ? 0 : sl.y;
            if (out_c) {
                out_c[3 * mi + 0] = first ? x0 : __int_as_float(sl.z);
                out_c[3 * mi + 1] = first ? y0 : __int_as_float(sl.w);
                out_c[3 * mi + 2] = first ? z0 : sz;
            }
        }
    };
    // Single wave: iteration m is kept in lane m % 64 and written 64
    // iterations at a time (one coalesced store instead of one single-lane
    // store per iteration).
    int keep_i = 0;
    float keep_x = cx, keep_y = cy, keep_z = cz;
    auto flush = [&](int m_last) {   // iterations (m_last & ~63) .. m_last
        const int m0 = m_last & ~63;
        if (m0 + lane <= m_last) {
            out_idx[m0 + lane] = keep_i;
            if (out_c) {
                out_c[3 * (m0 + lane) + 0] = keep_x;
                out_c[3 * (m0 + lane) + 1] = keep_y;
                out_c[3 * (m0 + lane) + 2] = keep_z;
            }
        }
    };

    // one iteration: the update, the wave and block reductions, the new centroid
    auto step = [&](int m) {
        // 1. distance to the newest centroid, running min, this thread's max
        int tmax = INT32_MIN;
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
            // both operands are >= 0 or the -1 sentinel, never NaN, so a
            // signed-int min on the bits is the strict-less running minimum
            // (one instruction; fminf would also canonicalize)
            const int nm = min(__float_as_int(dist3(x, y, z, cx, cy, cz)), __float_as_int(dm[q]));
            dm[q] = __int_as_float(nm);
            tmax = max(tmax, nm);
        }
        // 2. wave max; the lowest lane holding it; that lane's lowest slot.
        //    Every lane finds the lowest of its slots holding its own
        //    maximum while the wave maximum is reduced (the selects fill
        //    the DPP chain's latency), and the winning lane's answer is
        //    read out: the slot and the lane are wave-uniform, so only the
        //    winning lane's point is read.
        int ls = P - 1;
#pragma unroll
        for (int q = P - 2; q >= 0; --q) ls = __float_as_int(dm[q]) == tmax ? q : ls;
        const int wmax = wave_max_i32(tmax);
        const int wl = __builtin_ctzll(ballot(tmax == wmax));
        const int sq = __builtin_amdgcn_readlane(ls, wl);
        float sx, sy, sz;
        if constexpr (REG_XYZ) {
            sx = px[sq];   // wave-uniform index into the register arrays
            sy = py[sq];
            sz = pz[sq];
        } else {
            const int j = min(base + sq, N - 1);
            sx = p[3 * j + 0];
            sy = p[3 * j + 1];
            sz = p[3 * j + 2];
        }
        int sel;
        if constexpr (W == 1) {
            sel = __builtin_amdgcn_readlane(base + sq, wl);
            cx = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(sx), wl));
            cy = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(sy), wl));
            cz = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(sz), wl));
        } else {
            const int buf = m & (R - 1);
            if (lane == wl) {
                s_slot[buf][wave] = make_int4(wmax, base + sq, __float_as_int(sx), __float_as_int(sy));
                s_z[buf][wave] = sz;
            }
            __syncthreads();
            // 3. block winner: lane w < W inspects wave w's slot
            int4 sl = make_int4(INT32_MIN, 0, 0, 0);
            float slz = 0.0f;
            if (lane < W) {
                sl = s_slot[buf][lane];
                slz = s_z[buf][lane];
            }
            int gm;
            if constexpr (W <= 4) gm = __builtin_amdgcn_readlane(quad_max_i32(sl.x), 0);
            else if constexpr (W <= 8) gm = __builtin_amdgcn_readlane(oct_max_i32(sl.x), 7);
            else gm = __builtin_amdgcn_readlane(row_max_i32(sl.x), 0);
            const int ww = __builtin_ctzll(ballot(sl.x == gm));
            sel = __builtin_amdgcn_readlane(sl.y, ww);
            cx = __int_as_float(__builtin_amdgcn_readlane(sl.z, ww));
            cy = __int_as_float(__builtin_amdgcn_readlane(sl.w, ww));
            cz = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(slz), ww));
        }
        if constexpr (W == 1) {
            const bool mine = lane == (m & 63);
            keep_i = mine ? sel : keep_i;
            keep_x = mine ? cx : keep_x;
            keep_y = mine ? cy : keep_y;
            keep_z = mine ? cz : keep_z;
        } else {
            (void)sel;
        }
    };
    auto write_block = [&](int m_last) {
        if constexpr (W == 1) flush(m_last);
        else resolve(m_last);
    };
    if constexpr (P <= 4) {
        // blocks of 64 iterations with the results written after each
        // block: no per-iteration test (a few percent at small P)
        for (int mb = 1; mb < M;) {
            const int me = min(M, (mb | 63) + 1);
            for (int m = mb; m < me; ++m) step(m);
            if (wave == 0) write_block(me - 1);
            mb = me;
        }
        if (M == 1 && wave == 0) write_block(0);
    } else {
        // one flat loop (the blocked form schedules worse at large P)
        for (int m = 1; m < M; ++m) {
            step(m);
            if (wave == 0 && (m & 63) == 63) write_block(m);
        }
        if (wave == 0 && ((M - 1) & 63) != 63) write_block(M - 1);
    }
}

// Clouds of 513 to 8192 points: a copy of the cloud's coordinates in LDS.
// A wave's winner is then published as (distance bits, index) -- by lane
// 0, both values being wave-uniform -- and after the block reduction every
// wave reads the new centroid's coordinates from LDS at the winning index
// (one broadcast read), instead of the winning lane selecting them among
// its P register slots before the barrier (a chain of selects on the
// iteration's critical path: 15 % of an iteration at 4096 points, 27 % at
// 8192).  Everything else -- the update, the wave reduction, the slot search, the
// ring of per-wave winners resolved every 64 iterations -- is as in
// fps_kernel.
template <int T, int P>
__global__ __launch_bounds__(T) void fps_lds_kernel(const float* __restrict__ xyz, int N, int M,
                                                    int32_t* __restrict__ idx, float* __restrict__ cxyz) {
    constexpr int W = T / 64;
    constexpr int R = 128;                 // ring rows (two result blocks of 64 iterations)
    constexpr int NC = 3;                  // coordinates per point held in LDS
    __shared__ int2 s_slot[R][W];          // per-wave winner of iteration m in row m % R: distance bits, index
    __shared__ float s_c[T * P * NC];

    const int b = blockIdx.x;
    const float* __restrict__ p = xyz + (int64_t)b * N * 3;
    int32_t* __restrict__ out_idx = idx + (int64_t)b * M;
    float* __restrict__ out_c = cxyz ? cxyz + (int64_t)b * M * 3 : nullptr;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int base = tid * P;

    float px[P], py[P], pz[P], dm[P];
#pragma unroll
    for (int q = 0; q < P; ++q) {
        const int j = base + q;
        const bool ok = j < N;
        px[q] = ok ? p[3 * j + 0] : 0.0f;
        py[q] = ok ? p[3 * j + 1] : 0.0f;
        pz[q] = ok ? p[3 * j + 2] : 0.0f;
        dm[q] = ok ? __builtin_huge_valf() : -1.0f;  // +inf for real points; -1 never wins
        s_c[NC * j + 0] = px[q];
        s_c[NC * j + 1] = py[q];
        s_c[NC * j + 2] = pz[q];
    }
    __syncthreads();
    float cx = p[0], cy = p[1], cz = p[2];

    // lane l of wave 0 resolves iteration (m_last & ~63) + l from the ring
    // and stores it (iteration 0 is point 0)
    auto resolve = [&](int m_last) {
        const int mi = (m_last & ~63) + lane;
        const int row = mi & (R - 1);
        int best = s_slot[row][0].x, bw = 0;
#pragma unroll
        for (int w = 1; w < W; ++w) {
            const int d = s_slot[row][w].x;
            bw = d > best ? w : bw;
            best = d > best ? d : best;
        }
        if (mi <= m_last) {
            const bool first = mi == 0;
            const int sel = first ? 0 : s_slot[row][bw].y;
            out_idx[mi] = sel;
            if (out_c) {
                out_c[3 * mi + 0] = s_c[NC * sel + 0];
                out_c[3 * mi + 1] = s_c[NC * sel + 1];
                out_c[3 * mi + 2] = s_c[NC * sel + 2];
            }
        }
    };

    for (int m = 1; m < M; ++m) {
        // 1. distance to the newest centroid, running min, this thread's max
        int tmax = INT32_MIN;
#pragma unroll
        for (int q = 0; q < P; ++q) {
            const int nm = min(__float_as_int(dist3(px[q], py[q], pz[q], cx, cy, cz)), __float_as_int(dm[q]));
            dm[q] = __int_as_float(nm);
            tmax = max(tmax, nm);
        }
        // 2. wave max, the lowest lane holding it, that lane's lowest slot
        //    (each lane's lowest slot holding its own maximum, found while
        //    the wave maximum is reduced)
        int ls = P - 1;
#pragma unroll
        for (int q = P - 2; q >= 0; --q) ls = __float_as_int(dm[q]) == tmax ? q : ls;
        const int wmax = wave_max_i32(tmax);
        const int wl = __builtin_ctzll(ballot(tmax == wmax));
        const int sq = __builtin_amdgcn_readlane(ls, wl);
        const int buf = m & (R - 1);
        if (lane == 0) s_slot[buf][wave] = make_int2(wmax, wave * 64 * P + wl * P + sq);
        __syncthreads();
        // 3. block winner: lane w < W inspects wave w's slot; the new
        //    centroid's coordinates from LDS
        int2 sl = make_int2(INT32_MIN, 0);
        if (lane < W) sl = s_slot[buf][lane];
        int gm;
        if constexpr (W <= 8) gm = __builtin_amdgcn_readlane(oct_max_i32(sl.x), 7);
        else gm = __builtin_amdgcn_readlane(row_max_i32(sl.x), 0);
        const int ww = __builtin_ctzll(ballot(sl.x == gm));
        const int sel = __builtin_amdgcn_readlane(sl.y, ww);
        cx = s_c[NC * sel + 0];
        cy = s_c[NC * sel + 1];
        cz = s_c[NC * sel + 2];
        if (wave == 0 && (m & 63) == 63) resolve(m);
    }
    if (wave == 0 && ((M - 1) & 63) != 63) resolve(M - 1);
}

template <int T, int P>
static void launch_fps_lds(const float* xyz, int64_t B, int N, int M, int32_t* idx, float* cxyz, hipStream_t s) {
    static_assert(T >= 256 && T <= 1024 && T % 64 == 0, "4 to 16 waves");
    fps_lds_kernel<T, P><<<dim3((unsigned)B), dim3(T), 0, s>>>(xyz, N, M, idx, cxyz);
}


// ---------------------------------------------------------------------------
// Clouds of 8193 to 16384 points: spatial order and exact skipping.
//
// At 16 points per thread and four waves per SIMD the update of every
// running minimum is most of an iteration (VALU issue on the cloud's one
// CU), yet only the points near the newest centroid can change.  This form
// first puts the cloud in spatial order -- a counting sort of the points by
// the Morton code of their cell in a 16^3 grid over the cloud's box -- and
// gives thread t the P consecutive points [t P, t P + P) of that order, so
// each thread's points are close together.  Each thread keeps the box of its
// points; a wave skips the update when, for every one of its threads, a
// lower bound of the distance from the centroid to the thread's box is at
// least the thread's largest running minimum.  The bound is computed with
// the distance's own operations in the same order (dist3) on the per-axis
// gaps between the centroid and the box, max(lo - c, c - hi, 0): every
// operation is monotone in its operands and each gap is at most the
// corresponding |point - c| after rounding, so the bound never exceeds the
// distance the update would compute, and a skipped update is exactly the
// one that would have changed nothing.  Results are bit-identical to the
// other forms.
//
// Lowest index on ties: within a thread the points are sorted by original
// index at set-up, so the first slot holding the thread's maximum is its
// lowest; between lanes and between waves a tie is detected (two lanes or
// waves holding the maximum) and decided on the original index.  A wave's
// winner is published as (distance bits, position, original index, z); x
// and y of every position stay in LDS (the full coordinates of 16384 points
// would not fit beside the ring).
// ---------------------------------------------------------------------------

// Float min / max over the wave (all lanes active), uniform result.
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xf, 0xf, false));
}

__device__ __forceinline__ float wave_min_f32(float v) {
    v = fminf(v, dpp_f32<0x121>(v));
    v = fminf(v, dpp_f32<0x122>(v));
    v = fminf(v, dpp_f32<0x124>(v));
    v = fminf(v, dpp_f32<0x128>(v));
    v = fminf(v, __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v), 0x142, 0xa, 0xf, false)));
    v = fminf(v, __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v), 0x143, 0xc, 0xf, false)));
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}

__device__ __forceinline__ float wave_max_f32(float v) {
    v = fmaxf(v, dpp_f32<0x121>(v));
    v = fmaxf(v, dpp_f32<0x122>(v));
    v = fmaxf(v, dpp_f32<0x124>(v));
    v = fmaxf(v, dpp_f32<0x128>(v));
    v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v), 0x142, 0xa, 0xf, false)));
    v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v), 0x143, 0xc, 0xf, false)));
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}

// Int min over the wave (rare tie paths only).
__device__ __forceinline__ int wave_min_i32_shfl(int v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v = min(v, __shfl_xor(v, o));
    return v;
}

// 4-bit cell coordinate -> every third bit of a 12-bit Morton code.
__device__ __forceinline__ uint32_t morton_spread4(uint32_t v) {
    v &= 0xfu;
    v = (v | (v << 4)) & 0x0c3u;
    v = (v | (v << 2)) & 0x249u;
    return v;
}

template <int P>
struct RegVec {
    typedef float f32 __attribute__((ext_vector_type(P)));
    typedef int i32 __attribute__((ext_vector_type(P)));
};

template <int T, int P>
__global__ __launch_bounds__(T) void fps_skip_kernel(const float* __restrict__ xyz, int N, int M,
                                                     int32_t* __restrict__ idx, float* __restrict__ cxyz) {
    constexpr int W = T / 64;
    constexpr int NP = T * P;
    constexpr int R = 64;                // ring rows: two result blocks of 32 iterations
    constexpr int G = 16;                // grid cells per axis
    constexpr int NCELL = G * G * G;
    constexpr int CPT = NCELL / T;       // cells per thread in the scan
    static_assert(NCELL % T == 0 && NCELL <= NP && W <= 16, "shape");
    __shared__ float2 s_xy[NP];          // x, y of each position (set-up: the permutation, then the histogram)
    __shared__ int4 s_ring[R][W];        // wave winner of iteration m in row m % R: dist bits, position, index, z
    __shared__ float s_red[6][W];
    __shared__ int s_wsum[W];
    int* s_perm = reinterpret_cast<int*>(s_xy);
    int* s_hist = s_perm + NP;

    const int b = blockIdx.x;
    const float* __restrict__ p = xyz + (int64_t)b * N * 3;
    int32_t* __restrict__ out_idx = idx + (int64_t)b * M;
    float* __restrict__ out_c = cxyz ? cxyz + (int64_t)b * M * 3 : nullptr;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int base = tid * P;

    // z and the original indices are vectors: the winner's are read out with
    // a wave-uniform index (one indexed register move, not a select chain)
    float px[P], py[P], dm[P];
    typename RegVec<P>::f32 pz;
    typename RegVec<P>::i32 oi;   // original indices (the cell codes during the sort)
    {
        // 1. the cloud's box
        float mnx = __builtin_huge_valf(), mny = mnx, mnz = mnx, mxx = -mnx, mxy = -mnx, mxz = -mnx;
        for (int j = tid; j < N; j += T) {   // the points are read again for their cells
            const float x = p[3 * j + 0], y = p[3 * j + 1], z = p[3 * j + 2];
            mnx = fminf(mnx, x); mxx = fmaxf(mxx, x);
            mny = fminf(mny, y); mxy = fmaxf(mxy, y);
            mnz = fminf(mnz, z); mxz = fmaxf(mxz, z);
        }
        mnx = wave_min_f32(mnx); mny = wave_min_f32(mny); mnz = wave_min_f32(mnz);
        mxx = wave_max_f32(mxx); mxy = wave_max_f32(mxy); mxz = wave_max_f32(mxz);
        if (lane == 0) {
            s_red[0][wave] = mnx; s_red[1][wave] = mny; s_red[2][wave] = mnz;
            s_red[3][wave] = mxx; s_red[4][wave] = mxy; s_red[5][wave] = mxz;
        }
        for (int c = tid; c < NCELL; c += T) s_hist[c] = 0;
        __syncthreads();
#pragma unroll
        for (int w = 0; w < W; ++w) {
            mnx = fminf(mnx, s_red[0][w]); mny = fminf(mny, s_red[1][w]); mnz = fminf(mnz, s_red[2][w]);
            mxx = fmaxf(mxx, s_red[3][w]); mxy = fmaxf(mxy, s_red[4][w]); mxz = fmaxf(mxz, s_red[5][w]);
        }
        const float ix = mxx > mnx ? (float)G / (mxx - mnx) : 0.0f;
        const float iy = mxy > mny ? (float)G / (mxy - mny) : 0.0f;
        const float iz = mxz > mnz ? (float)G / (mxz - mnz) : 0.0f;
        // 2. cell histogram (the cell only orders the points: any cell,
        //    even of a non-finite coordinate, keeps the result exact)
#pragma unroll
        for (int q = 0; q < P; ++q) {
            const int j = tid + q * T;
            const int jj = j < N ? j : 0;
            const uint32_t gx = (uint32_t)fminf(fmaxf((p[3 * jj + 0] - mnx) * ix, 0.0f), (float)(G - 1));
            const uint32_t gy = (uint32_t)fminf(fmaxf((p[3 * jj + 1] - mny) * iy, 0.0f), (float)(G - 1));
            const uint32_t gz = (uint32_t)fminf(fmaxf((p[3 * jj + 2] - mnz) * iz, 0.0f), (float)(G - 1));
            oi[q] = (int)(morton_spread4(gx) | (morton_spread4(gy) << 1) | (morton_spread4(gz) << 2));
            if (j < N) atomicAdd(&s_hist[oi[q]], 1);
        }
        __syncthreads();
        // 3. exclusive scan of the counts
        int cnt[CPT], run = 0;
#pragma unroll
        for (int k = 0; k < CPT; ++k) {
            cnt[k] = s_hist[tid * CPT + k];
            run += cnt[k];
        }
        int incl = run;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int v = __shfl_up(incl, o);
            if (lane >= o) incl += v;
        }
        if (lane == 63) s_wsum[wave] = incl;
        __syncthreads();
        int off = incl - run;
        for (int w = 0; w < wave; ++w) off += s_wsum[w];
#pragma unroll
        for (int k = 0; k < CPT; ++k) {
            s_hist[tid * CPT + k] = off;
            off += cnt[k];
        }
        for (int j = N + tid; j < NP; j += T) s_perm[j] = INT32_MAX;   // padding positions
        __syncthreads();
        // 4. scatter the original indices into cell order
#pragma unroll
        for (int q = 0; q < P; ++q) {
            const int j = tid + q * T;
            if (j < N) s_perm[atomicAdd(&s_hist[oi[q]], 1)] = j;
        }
        __syncthreads();
        // 5. this thread's positions, ascending in original index
        //    (odd-even transposition sort)
#pragma unroll
        for (int q = 0; q < P; ++q) oi[q] = s_perm[base + q];
#pragma unroll
        for (int r = 0; r < P; ++r) {
#pragma unroll
            for (int q = r & 1; q + 1 < P; q += 2) {
                const int lo = min(oi[q], oi[q + 1]), hi = max(oi[q], oi[q + 1]);
                oi[q] = lo;
                oi[q + 1] = hi;
            }
        }
        __syncthreads();   // the permutation is read; its space becomes s_xy
    }
    float bnx = __builtin_huge_valf(), bny = bnx, bnz = bnx, bxx = -bnx, bxy = -bnx, bxz = -bnx;
#pragma unroll
    for (int q = 0; q < P; ++q) {
        const bool ok = oi[q] != INT32_MAX;
        const int j = ok ? oi[q] : 0;
        px[q] = ok ? p[3 * j + 0] : 0.0f;
        py[q] = ok ? p[3 * j + 1] : 0.0f;
        pz[q] = ok ? p[3 * j + 2] : 0.0f;
        dm[q] = ok ? __builtin_huge_valf() : -1.0f;   // +inf for real points; -1 never wins
        s_xy[base + q] = make_float2(px[q], py[q]);
        if (ok) {
            bnx = fminf(bnx, px[q]); bxx = fmaxf(bxx, px[q]);
            bny = fminf(bny, py[q]); bxy = fmaxf(bxy, py[q]);
            bnz = fminf(bnz, pz[q]); bxz = fmaxf(bxz, pz[q]);
        }
    }

    // this thread's largest running minimum; the wave's winner
    int tmax = 0, wmax = 0, wpos = 0, woi = 0;
    float wz = 0.0f;
    auto select = [&]() {
        tmax = __float_as_int(dm[0]);
#pragma unroll
        for (int q = 1; q < P; ++q) tmax = max(tmax, __float_as_int(dm[q]));
        int ls = P - 1;
#pragma unroll
        for (int q = P - 2; q >= 0; --q) ls = __float_as_int(dm[q]) == tmax ? q : ls;
        const int wm = wave_max_i32(tmax);
        const uint64_t tie = ballot(tmax == wm);
        int wl = __builtin_ctzll(tie);
        if (tie & (tie - 1)) {   // two lanes hold the maximum: the lower original index
            int lo = oi[P - 1];
#pragma unroll
            for (int q = P - 2; q >= 0; --q) lo = ls == q ? oi[q] : lo;
            const int key = tmax == wm ? lo : INT32_MAX;
            wl = __builtin_ctzll(ballot(key == wave_min_i32_shfl(key)));
        }
        const int sq = __builtin_amdgcn_readlane(ls, wl);
        wmax = wm;
        wpos = (wave * 64 + wl) * P + sq;
        woi = __builtin_amdgcn_readlane(oi[sq], wl);
        wz = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(pz[sq]), wl));
    };
    select();
    __syncthreads();   // s_xy complete

    const float x0 = p[0], y0 = p[1], z0 = p[2];
    float cx = x0, cy = y0, cz = z0;

    // lane l < 32 of wave 0 resolves iteration (m_last & ~31) + l from the
    // ring (highest distance, then lowest index) and stores it
    auto resolve = [&](int m_last) {
        if (lane < 32) {
            const int mi = (m_last & ~31) + lane;
            const int row = mi & (R - 1);
            int best = INT32_MIN, boi = INT32_MAX, bw = 0;
#pragma unroll
            for (int w = 0; w < W; ++w) {
                const int4 e = s_ring[row][w];
                const bool better = e.x > best || (e.x == best && e.z < boi);
                best = better ? e.x : best;
                boi = better ? e.z : boi;
                bw = better ? w : bw;
            }
            if (mi <= m_last) {
                const bool first = mi == 0;
                out_idx[mi] = first ? 0 : boi;
                if (out_c) {
                    const int4 e = s_ring[row][bw];
                    const float2 xy = s_xy[e.y];
                    out_c[3 * mi + 0] = first ? x0 : xy.x;
                    out_c[3 * mi + 1] = first ? y0 : xy.y;
                    out_c[3 * mi + 2] = first ? z0 : __int_as_float(e.w);
                }
            }
        }
    };

    for (int m = 1; m < M; ++m) {
        // 1. skip test against this thread's box, then the update
        const float gx = fmaxf(fmaxf(bnx - cx, cx - bxx), 0.0f);
        const float gy = fmaxf(fmaxf(bny - cy, cy - bxy), 0.0f);
        const float gz = fmaxf(fmaxf(bnz - cz, cz - bxz), 0.0f);
        float lb = gx * gx;
        lb = __builtin_fmaf(gy, gy, lb);
        lb = __builtin_fmaf(gz, gz, lb);
        if (ballot(__float_as_int(lb) < tmax)) {
#pragma unroll
            for (int q = 0; q < P; ++q)
                dm[q] = __int_as_float(
                    min(__float_as_int(dist3(px[q], py[q], pz[q], cx, cy, cz)), __float_as_int(dm[q])));
            select();
        }
        // 2. publish the wave's winner; block winner; the new centroid
        const int buf = m & (R - 1);
        if (lane == 0) s_ring[buf][wave] = make_int4(wmax, wpos, woi, __float_as_int(wz));
        __syncthreads();
        int4 e = make_int4(INT32_MIN, 0, INT32_MAX, 0);
        if (lane < W) e = s_ring[buf][lane];
        int gm;
        if constexpr (W <= 8) gm = __builtin_amdgcn_readlane(oct_max_i32(e.x), 7);
        else gm = __builtin_amdgcn_readlane(row_max_i32(e.x), 0);
        const uint64_t eq = ballot(e.x == gm) & ((1ull << W) - 1);
        int ww = __builtin_ctzll(eq);
        if (eq & (eq - 1)) {
            const int key = (lane < W && e.x == gm) ? e.z : INT32_MAX;
            ww = __builtin_ctzll(ballot(key == wave_min_i32_shfl(key)));
        }
        const int sel = __builtin_amdgcn_readlane(e.y, ww);
        cz = __int_as_float(__builtin_amdgcn_readlane(e.w, ww));
        const float2 xy = s_xy[sel];
        cx = xy.x;
        cy = xy.y;
        if (wave == 0 && (m & 31) == 31) resolve(m);
    }
    if (wave == 0 && ((M - 1) & 31) != 31) resolve(M - 1);
}

template <int T, int P>
static void launch_fps_skip(const float* xyz, int64_t B, int N, int M, int32_t* idx, float* cxyz, hipStream_t s) {
    fps_skip_kernel<T, P><<<dim3((unsigned)B), dim3(T), 0, s>>>(xyz, N, M, idx, cxyz);
}

template <int T, int P, bool REG>
static void launch_fps(const float* xyz, int64_t B, int N, int M, int32_t* idx, float* cxyz, hipStream_t s) {
    fps_kernel<T, P, REG><<<dim3((unsigned)B), dim3(T), 0, s>>>(xyz, N, M, idx, cxyz);
}

// ---------------------------------------------------------------------------
// Large clouds: G one-wave workgroups per cloud.
//
// One CU's vector ALUs bound the single-workgroup kernel once every thread
// holds 16 points (16384-point clouds: about 1.3 us per iteration when every
// point is updated, 0.8 us with the skipping of fps_skip_kernel).  Here
// the points are spread over G single-wave workgroups (workgroup g owns the
// contiguous points [64 P g, 64 P (g + 1)), lane l the P points from
// 64 P g + P l), so an iteration's update is P points per lane on G CUs,
// and the workgroups exchange their local winners through global memory:
//  * the workspace holds, per cloud, 2 x G slots of four 64-bit words,
//    cleared by a fill kernel before the launch;
//  * at iteration m each workgroup stores its winner in slot [m % 2][g]:
//    word 0 = m << 48 | distance bits << 16 | index, words 1-3 = m << 32 |
//    x, y, z bits.  Every word carries the tag m, so a reader accepts a
//    slot only when all four words belong to iteration m, whatever order
//    the stores land in (aligned 64-bit accesses are single-copy atomic);
//  * lane h < G of every workgroup polls slot [m % 2][h] (agent-scope
//    atomic loads) until all G carry tag m, then the largest distance wins
//    and, on ties, the lowest h -- workgroups order the indices, so that is
//    the lowest index, as in the sequential rule;
//  * a workgroup publishes iteration m + 2 into the same parity only after
//    reading every slot of iteration m + 1, which each workgroup writes
//    only after reading all of iteration m: two parities never lose a
//    value, and a cleared slot (tag 0) never matches m >= 1.
// Every wait is bounded: after kFpsSpinCap polls the workgroup sets the
// error word in the workspace and continues alone with its local winners
// (valid indices, wrong results), so the kernel always drains.  Waiting
// needs the cloud's G workgroups resident at once; a launch has at most
// 8 x ceil(B / 8) x 64 single-wave workgroups, which fit on the chip beside
// any other kernel's workgroups (those finish without waiting on this one).
// Workgroups of one cloud are numbered congruent modulo 8 so that the
// round-robin dispatch puts them on one XCD and their slots in one L2;
// correctness does not depend on that placement.
// ---------------------------------------------------------------------------

constexpr int kFpsMaxGroups = 64;   // one polling lane per group
constexpr int kFpsSpinCap = 1 << 20;
constexpr size_t kFpsWsHeader = 256;   // error word, then the slots

__global__ void fps_clear_kernel(uint64_t* __restrict__ w, int64_t n) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        w[i] = 0;
}

__device__ __forceinline__ void ws_store(uint64_t* p, uint64_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t ws_load(const uint64_t* p) {
    return __hip_atomic_load(const_cast<uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <int P>
__global__ __launch_bounds__(64) void fps_multi_kernel(const float* __restrict__ xyz, int B, int N, int M, int G,
                                                       int32_t* __restrict__ idx, float* __restrict__ cxyz,
                                                       uint64_t* __restrict__ slots, unsigned* __restrict__ err) {
    // blockIdx -> (cloud, group): ids congruent mod 8 share a cloud
    const int i = blockIdx.x;
    const int xcd = i & 7, k = i >> 3;
    const int b = xcd + 8 * (k / G);
    const int g = k - (k / G) * G;
    if (b >= B) return;
    const int lane = threadIdx.x;
    const float* __restrict__ p = xyz + (int64_t)b * N * 3;
    const int base = g * 64 * P + lane * P;
    uint64_t* __restrict__ cs = slots + (int64_t)b * 2 * G * 4;   // this cloud's [2][G][4] words

    float px[P], py[P], pz[P], dm[P];
#pragma unroll
    for (int q = 0; q < P; ++q) {
        const int j = base + q;
        const bool ok = j < N;
        px[q] = ok ? p[3 * j + 0] : 0.0f;
        py[q] = ok ? p[3 * j + 1] : 0.0f;
        pz[q] = ok ? p[3 * j + 2] : 0.0f;
        dm[q] = ok ? __builtin_huge_valf() : -1.0f;   // -1 never wins
    }
    float cx = p[0], cy = p[1], cz = p[2];
    // workgroup 0 records the results: iteration m in lane m % 64, stored
    // 64 iterations at a time
    int keep_i = 0;
    float keep_x = cx, keep_y = cy, keep_z = cz;
    int32_t* __restrict__ out_idx = idx + (int64_t)b * M;
    float* __restrict__ out_c = cxyz ? cxyz + (int64_t)b * M * 3 : nullptr;
    auto flush = [&](int m_last) {
        const int m0 = m_last & ~63;
        if (m0 + lane <= m_last) {
            out_idx[m0 + lane] = keep_i;
            if (out_c) {
                out_c[3 * (m0 + lane) + 0] = keep_x;
                out_c[3 * (m0 + lane) + 1] = keep_y;
                out_c[3 * (m0 + lane) + 2] = keep_z;
            }
        }
    };
    bool alone = false;   // set once a wait hit the cap

    for (int m = 1; m < M; ++m) {
        // 1. running minima and this lane's largest (signed-int min/max on
        //    the bits: values are >= 0 or the -1 sentinel)
        int tmax = INT32_MIN;
#pragma unroll
        for (int q = 0; q < P; ++q) {
            const int nm = min(__float_as_int(dist3(px[q], py[q], pz[q], cx, cy, cz)), __float_as_int(dm[q]));
            dm[q] = __int_as_float(nm);
            tmax = max(tmax, nm);
        }
        // 2. local winner: the lowest lane holding the max, its lowest slot
        const int wmax = wave_max_i32(tmax);
        const int wl = __builtin_ctzll(ballot(tmax == wmax));
        int sq = P - 1;
#pragma unroll
        for (int q = P - 1; q >= 0; --q) {
            const uint64_t hold = ballot(__float_as_int(dm[q]) == wmax);
            sq = ((hold >> wl) & 1ull) ? q : sq;
        }
        sq = __builtin_amdgcn_readfirstlane(sq);
        const int lj = __builtin_amdgcn_readlane(base + sq, wl);
        const int lx = __builtin_amdgcn_readlane(__float_as_int(px[sq]), wl);
        const int ly = __builtin_amdgcn_readlane(__float_as_int(py[sq]), wl);
        const int lz = __builtin_amdgcn_readlane(__float_as_int(pz[sq]), wl);
        int sel = lj;
        int sx = lx, sy = ly, sz = lz;
        if (!alone) {
            // 3. publish (every workgroup holds a real point, so wmax >= 0)
            uint64_t* mine = cs + ((m & 1) * G + g) * 4;
            const uint64_t tag = (uint64_t)m;
            if (lane == 0) {
                ws_store(mine + 0, (tag << 48) | ((uint64_t)(uint32_t)wmax << 16) | (uint64_t)(uint32_t)lj);
                ws_store(mine + 1, (tag << 32) | (uint32_t)lx);
                ws_store(mine + 2, (tag << 32) | (uint32_t)ly);
                ws_store(mine + 3, (tag << 32) | (uint32_t)lz);
            }
            // 4. wait for all G slots of iteration m (lane h reads slot h)
            const uint64_t* theirs = cs + ((m & 1) * G + min(lane, G - 1)) * 4;
            uint64_t w0 = 0, w1 = 0, w2 = 0, w3 = 0;
            bool ok = lane >= G;
            for (int spins = 0;; ++spins) {
                if (!ok) {
                    w0 = ws_load(theirs + 0);
                    w1 = ws_load(theirs + 1);
                    w2 = ws_load(theirs + 2);
                    w3 = ws_load(theirs + 3);
                    ok = (w0 >> 48) == tag && (w1 >> 32) == tag && (w2 >> 32) == tag && (w3 >> 32) == tag;
                }
                if (ballot(!ok) == 0ull) break;
                if (spins >= kFpsSpinCap) {
                    alone = true;
                    if (lane == 0) atomicOr(err, 1u);
                    break;
                }
            }
            if (!alone) {
                // 5. global winner: the largest distance, then the lowest group
                const int d = lane < G ? (int)((w0 >> 16) & 0x7fffffffull) : INT32_MIN;
                const int gmax = wave_max_i32(d);
                const int ww = __builtin_ctzll(ballot(d == gmax));
                sel = __builtin_amdgcn_readlane((int)(w0 & 0xffffull), ww);
                sx = __builtin_amdgcn_readlane((int)(uint32_t)w1, ww);
                sy = __builtin_amdgcn_readlane((int)(uint32_t)w2, ww);
                sz = __builtin_amdgcn_readlane((int)(uint32_t)w3, ww);
            }
        }
        cx = __int_as_float(sx);
        cy = __int_as_float(sy);
        cz = __int_as_float(sz);
        if (g == 0) {
            const bool keep = lane == (m & 63);
            keep_i = keep ? sel : keep_i;
            keep_x = keep ? cx : keep_x;
            keep_y = keep ? cy : keep_y;
            keep_z = keep ? cz : keep_z;
            if ((m & 63) == 63) flush(m);
        }
    }
    if (g == 0 && ((M - 1) & 63) != 63) flush(M - 1);
}

// Shape of the multi-workgroup form: P points per lane, G workgroups per
// cloud (every workgroup holds at least one real point).
struct FpsMultiPlan {
    int P, G;
};
static FpsMultiPlan fps_multi_plan(int64_t N) {
    const int P = N <= 8192 ? 4 : (N <= 16384 ? 8 : 16);
    return {P, (int)ceil_div(N, 64 * P)};
}
// The multi-workgroup form runs for clouds above 32768 points, where the
// single-workgroup kernel can no longer keep the coordinates in registers
// and re-reads the cloud every iteration (65536 points: 17.5 us per
// iteration there, 4.6 us here).  Below, one exchange through global memory
// (about 0.7 us for one tagged word between CUs, 2-2.5 us for this
// kernel's four-word slots, measured on MI355X) costs more than a whole
// single-workgroup iteration (0.46 us at 4096 points, 0.8 us at 16384 with
// skipping, 2.66 us at 32768 against 2.72 us here).
constexpr int64_t kFpsMultiMinN = 32769;

static bool fps_use_multi(int64_t N, int64_t M) {
    return N >= kFpsMultiMinN && M >= 2 && fps_multi_plan(N).G <= kFpsMaxGroups;
}

static size_t fps_ws_bytes(int64_t B, int64_t N, int64_t M) {
    if (B <= 0 || !fps_use_multi(N, M)) return 0;
    return kFpsWsHeader + (size_t)B * 2 * fps_multi_plan(N).G * 4 * sizeof(uint64_t);
}

template <int P>
static int launch_fps_multi(const float* xyz, int64_t B, int N, int M, int G, int32_t* idx, float* cxyz, void* ws,
                            hipStream_t s) {
    uint64_t* slots = reinterpret_cast<uint64_t*>(static_cast<char*>(ws) + kFpsWsHeader);
    unsigned* err = static_cast<unsigned*>(ws);
    const int64_t words = (int64_t)B * 2 * G * 4;
    const int64_t clear = words + kFpsWsHeader / 8;
    fps_clear_kernel<<<dim3((unsigned)std::min<int64_t>(ceil_div(clear, 256), 1024)), dim3(256), 0, s>>>(
        static_cast<uint64_t*>(ws), clear);
    int rc = after_launch("mesorasi_fps");
    if (rc != MESORASI_OK) return rc;
    const int64_t grid = 8 * ceil_div(B, 8) * G;
    fps_multi_kernel<P><<<dim3((unsigned)grid), dim3(64), 0, s>>>(xyz, (int)B, N, M, G, idx, cxyz, slots, err);
    return after_launch("mesorasi_fps");
}

// Sampling of an already sampled, ordered set: the first M points of that
// order (one thread per output point and coordinate triple).
__global__ __launch_bounds__(256) void fps_prefix_kernel(const int32_t* __restrict__ idx_prev,
                                                        const float* __restrict__ cxyz_prev, int64_t B, int Mp, int M,
                                                        int32_t* __restrict__ idx, float* __restrict__ cxyz) {
    const int64_t total = B * M;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t b = e / M;
        const int k = (int)(e - b * M);
        const int64_t src = b * Mp + k;
        // a step whose largest min-distance was 0 took point 0 in the earlier
        // run (index 0 there) and takes subset point 0 here
        idx[e] = (k == 0 || idx_prev[src] != 0) ? k : 0;
        if (cxyz) {
            cxyz[3 * e + 0] = cxyz_prev[3 * src + 0];
            cxyz[3 * e + 1] = cxyz_prev[3 * src + 1];
            cxyz[3 * e + 2] = cxyz_prev[3 * src + 2];
        }
    }
}

// Several nested levels in one launch: level v takes the first M[v] points
// of level 0's sampling (the prefix of a prefix is a prefix, and the index
// rule depends only on level 0's indices).  Thread e of the flattened
// (level, cloud, k) range writes one point.
struct FpsLevels {
    int n;
    int M[MESORASI_MAX_LAYERS];
    int64_t start[MESORASI_MAX_LAYERS + 1];   // flattened offsets of the levels
    int32_t* idx[MESORASI_MAX_LAYERS];
    float* cxyz[MESORASI_MAX_LAYERS];
};

__global__ __launch_bounds__(256) void fps_prefix_levels_kernel(const int32_t* __restrict__ idx0,
                                                               const float* __restrict__ cxyz0, int64_t B, int M0,
                                                               FpsLevels lv) {
    const int64_t total = lv.start[lv.n];
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
        int v = 0;
        while (e >= lv.start[v + 1]) ++v;
        const int64_t r = e - lv.start[v];
        const int M = lv.M[v];
        const int64_t b = r / M;
        const int k = (int)(r - b * M);
        const int64_t src = b * M0 + k;
        lv.idx[v][r] = (k == 0 || idx0[src] != 0) ? k : 0;
        if (lv.cxyz[v]) {
            lv.cxyz[v][3 * r + 0] = cxyz0[3 * src + 0];
            lv.cxyz[v][3 * r + 1] = cxyz0[3 * src + 1];
            lv.cxyz[v][3 * r + 2] = cxyz0[3 * src + 2];
        }
    }
}

}  // namespace meso

using namespace meso;

extern "C" size_t mesorasi_fps_workspace(int64_t B, int64_t N, int64_t M) {
    if (B < 0 || N < 0 || M < 0 || M > N || N > MESORASI_MAX_N_FPS) return 0;
    return fps_ws_bytes(B, N, M);
}

extern "C" int mesorasi_fps(const float* xyz, int64_t B, int64_t N, int64_t M, int32_t* idx, float* cxyz, void* ws,
                            size_t ws_bytes, void* stream) {
    MESO_REQUIRE(B >= 0 && N >= 0 && M >= 0, MESORASI_EINVAL, "mesorasi_fps: negative size (B=%lld N=%lld M=%lld)",
                 (long long)B, (long long)N, (long long)M);
    MESO_REQUIRE(M <= N, MESORASI_EINVAL, "mesorasi_fps: M = %lld > N = %lld", (long long)M, (long long)N);
    if (B == 0 || M == 0) return MESORASI_OK;
    MESO_REQUIRE(xyz && idx, MESORASI_EINVAL, "mesorasi_fps: NULL xyz or idx");
    MESO_REQUIRE(N <= MESORASI_MAX_N_FPS, MESORASI_EUNSUPPORTED, "mesorasi_fps: N = %lld > %d", (long long)N,
                 MESORASI_MAX_N_FPS);
    MESO_REQUIRE(B <= 0x7fffffff, MESORASI_EUNSUPPORTED, "mesorasi_fps: B too large");
    const size_t need = fps_ws_bytes(B, N, M);
    MESO_REQUIRE(ws_bytes >= need && (need == 0 || ws), MESORASI_EWORKSPACE, "mesorasi_fps: workspace %zu < %zu bytes",
                 ws_bytes, need);
    MESO_REQUIRE(need == 0 || aligned(ws, 8), MESORASI_EINVAL, "mesorasi_fps: workspace not 8-byte aligned");
    hipStream_t s = as_stream(stream);
    const int n = (int)N, m = (int)M;
    if (need > 0) {
        const FpsMultiPlan pl = fps_multi_plan(N);
        if (pl.P == 4) return launch_fps_multi<4>(xyz, B, n, m, pl.G, idx, cxyz, ws, s);
        if (pl.P == 8) return launch_fps_multi<8>(xyz, B, n, m, pl.G, idx, cxyz, ws, s);
        return launch_fps_multi<16>(xyz, B, n, m, pl.G, idx, cxyz, ws, s);
    }
    // workgroup shape per cloud size, from a sweep on MI355X: the iteration
    // time is a fixed reduction/barrier chain plus P points of VALU work
    if (n <= 128) launch_fps<64, 2, true>(xyz, B, n, m, idx, cxyz, s);
    else if (n <= 256) launch_fps<64, 4, true>(xyz, B, n, m, idx, cxyz, s);
    else if (n <= 512) launch_fps<256, 2, true>(xyz, B, n, m, idx, cxyz, s);
    else if (n <= 1024) launch_fps_lds<256, 4>(xyz, B, n, m, idx, cxyz, s);
    else if (n <= 2048) launch_fps_lds<512, 4>(xyz, B, n, m, idx, cxyz, s);
    else if (n <= 4096) launch_fps_lds<512, 8>(xyz, B, n, m, idx, cxyz, s);
    else if (n <= 8192) launch_fps_lds<1024, 8>(xyz, B, n, m, idx, cxyz, s);
    else if (n <= 16384) launch_fps_skip<1024, 16>(xyz, B, n, m, idx, cxyz, s);
    else if (n <= 32768) launch_fps<1024, 32, false>(xyz, B, n, m, idx, cxyz, s);
    else launch_fps<1024, 64, false>(xyz, B, n, m, idx, cxyz, s);
    return after_launch("mesorasi_fps");
}

extern "C" int mesorasi_fps_prefix(const int32_t* idx_prev, const float* cxyz_prev, int64_t B, int64_t M_prev,
                                   int64_t M, int32_t* idx, float* cxyz, void* stream) {
    MESO_REQUIRE(B >= 0 && M_prev >= 0 && M >= 0, MESORASI_EINVAL,
                 "mesorasi_fps_prefix: negative size (B=%lld M_prev=%lld M=%lld)", (long long)B, (long long)M_prev,
                 (long long)M);
    MESO_REQUIRE(M <= M_prev, MESORASI_EINVAL, "mesorasi_fps_prefix: M = %lld > M_prev = %lld", (long long)M,
                 (long long)M_prev);
    if (B == 0 || M == 0) return MESORASI_OK;
    MESO_REQUIRE(idx_prev && idx, MESORASI_EINVAL, "mesorasi_fps_prefix: NULL idx_prev or idx");
    MESO_REQUIRE(!cxyz || cxyz_prev, MESORASI_EINVAL, "mesorasi_fps_prefix: cxyz requested without cxyz_prev");
    MESO_REQUIRE(M_prev <= MESORASI_MAX_N_FPS, MESORASI_EUNSUPPORTED, "mesorasi_fps_prefix: M_prev = %lld > %d",
                 (long long)M_prev, MESORASI_MAX_N_FPS);
    MESO_REQUIRE(B <= 0x7fffffff, MESORASI_EUNSUPPORTED, "mesorasi_fps_prefix: B too large");
    const int64_t total = B * M;
    const unsigned grid = (unsigned)std::min<int64_t>(ceil_div(total, 256), 4096);
    fps_prefix_kernel<<<dim3(grid), dim3(256), 0, as_stream(stream)>>>(idx_prev, cxyz_prev, B, (int)M_prev, (int)M,
                                                                       idx, cxyz);
    return after_launch("mesorasi_fps_prefix");
}

extern "C" int mesorasi_fps_prefix_levels(const int32_t* idx0, const float* cxyz0, int64_t B, int64_t M0,
                                          int32_t n_levels, const int64_t* M, int32_t* const* idx,
                                          float* const* cxyz, void* stream) {
    const char* who = "mesorasi_fps_prefix_levels";
    MESO_REQUIRE(B >= 0 && M0 >= 0, MESORASI_EINVAL, "%s: negative size", who);
    MESO_REQUIRE(n_levels >= 0 && n_levels <= MESORASI_MAX_LAYERS, MESORASI_EINVAL, "%s: n_levels = %d", who,
                 n_levels);
    MESO_REQUIRE(n_levels == 0 || (M && idx), MESORASI_EINVAL, "%s: NULL M or idx", who);
    MESO_REQUIRE(M0 <= MESORASI_MAX_N_FPS, MESORASI_EUNSUPPORTED, "%s: M0 = %lld > %d", who, (long long)M0,
                 MESORASI_MAX_N_FPS);
    MESO_REQUIRE(B <= 0x7fffffff, MESORASI_EUNSUPPORTED, "%s: B too large", who);
    FpsLevels lv{};
    lv.n = n_levels;
    int64_t total = 0;
    bool any_xyz = false;
    for (int v = 0; v < n_levels; ++v) {
        MESO_REQUIRE(M[v] >= 0 && M[v] <= M0, MESORASI_EINVAL, "%s: M[%d] = %lld outside [0, M0 = %lld]", who, v,
                     (long long)M[v], (long long)M0);
        lv.M[v] = (int)M[v];
        lv.start[v] = total;
        total += B * M[v];
        lv.idx[v] = idx[v];
        lv.cxyz[v] = cxyz ? cxyz[v] : nullptr;
        MESO_REQUIRE(B * M[v] == 0 || idx[v], MESORASI_EINVAL, "%s: NULL idx[%d]", who, v);
        any_xyz = any_xyz || (lv.cxyz[v] && B * M[v] > 0);
    }
    lv.start[n_levels] = total;
    if (total == 0) return MESORASI_OK;
    MESO_REQUIRE(idx0, MESORASI_EINVAL, "%s: NULL idx0", who);
    MESO_REQUIRE(!any_xyz || cxyz0, MESORASI_EINVAL, "%s: cxyz requested without cxyz0", who);
    const unsigned grid = (unsigned)std::min<int64_t>(ceil_div(total, 256), 4096);
    fps_prefix_levels_kernel<<<dim3(grid), dim3(256), 0, as_stream(stream)>>>(idx0, cxyz0, B, (int)M0, lv);
    return after_launch(who);
}

// Ball query on gfx950 -- the neighbor search N (Sec. 3.1 "Neighbor Search")
// that fills the neighbor index table (NIT, Sec. 4.1 walk-through).
//
// One wave per query.  The wave walks the cloud in 64-point chunks in index
// order, eight chunks per step (coordinates fetched together, every chunk's
// test and ballot formed before its hits are placed); each lane tests one
// point, a ballot collects the chunk's hits and mbcnt gives every hit its
// rank, so hits land in ascending index order with no sorting.  The walk
// stops after the step that completes K hits (the early exit is what makes
// dense surface-like clouds cheap), then the tail of the row is padded with
// the first hit.  Clouds of 2048 to 8191 points are first copied into LDS
// by a workgroup that serves 16 queries; from 8192 points a grid of cells
// bounds the candidates.
#include <algorithm>
#include <cmath>

#include "common.h"

namespace meso {

constexpr int kBqWaves = 4;
constexpr int kBqChunks = 8;   // 64-point chunks per walk step

// The index-order walk of one query by one wave: fills row[0 .. K) and
// returns the number of real hits (<= K).  pt(j, x, y, z) reads point j
// (from memory, or from the LDS copy of the cloud).
template <class PT>
__device__ __forceinline__ int bq_walk(PT pt, int N, float qx, float qy, float qz, float r2, int K,
                                       int32_t* __restrict__ row, int lane) {
    int n = 0;
    int first = 0;
    for (int base0 = 0; base0 < N && n < K; base0 += 64 * kBqChunks) {
        // kBqChunks chunks per step, straight-line: the coordinates are
        // requested together (lanes past N read point N - 1 and never hit)
        // and every chunk's test and ballot is formed before the hits are
        // placed, in index order; hits past the K-th are counted but not
        // stored, and the walk stops after the step that completes K
        float cx[kBqChunks], cy[kBqChunks], cz[kBqChunks];
#pragma unroll
        for (int u = 0; u < kBqChunks; ++u) pt(min(base0 + 64 * u + lane, N - 1), cx[u], cy[u], cz[u]);
        bool hit[kBqChunks];
        uint64_t mask[kBqChunks];
#pragma unroll
        for (int u = 0; u < kBqChunks; ++u) {
            hit[u] = base0 + 64 * u + lane < N && dist3(cx[u], cy[u], cz[u], qx, qy, qz) < r2;
            mask[u] = ballot(hit[u]);
        }
#pragma unroll
        for (int u = 0; u < kBqChunks; ++u) {
            if (mask[u]) {
                const int base = base0 + 64 * u;
                if (n == 0) first = base + __builtin_ctzll(mask[u]);
                const int pos = n + mask_rank(mask[u]);
                if (hit[u] && pos < K) row[pos] = base + lane;
                n += __builtin_popcountll(mask[u]);
            }
        }
    }
    n = min(n, K);
    const int pad = n > 0 ? first : 0;
    for (int k = n + lane; k < K; k += 64) row[k] = pad;
    return n;
}

__global__ __launch_bounds__(64 * kBqWaves) void ball_query_kernel(const float* __restrict__ xyz,
                                                                   const float* __restrict__ qxyz, int64_t BM, int N,
                                                                   int M, float r2, int K, int32_t* __restrict__ nit,
                                                                   int32_t* __restrict__ cnt) {
    const int64_t gq = (int64_t)blockIdx.x * kBqWaves + (threadIdx.x >> 6);
    if (gq >= BM) return;  // whole wave leaves together; no barriers below
    const int lane = threadIdx.x & 63;
    const int64_t b = gq / M;
    const float* __restrict__ p = xyz + b * (int64_t)N * 3;
    auto pt = [&](int j, float& x, float& y, float& z) {
        x = p[3 * j + 0];
        y = p[3 * j + 1];
        z = p[3 * j + 2];
    };
    const int n = bq_walk(pt, N, qxyz[gq * 3 + 0], qxyz[gq * 3 + 1], qxyz[gq * 3 + 2], r2, K, nit + gq * K, lane);
    if (cnt && lane == 0) cnt[gq] = n;
}

// Mid-size clouds (kBqLdsMinN .. kBqGridMinN - 1 points): a workgroup of
// kBqLdsWaves waves serves as many queries of one cloud and first copies
// the cloud into LDS (coordinate planes x, y, z).  Surface-like clouds at
// small radii leave most balls short of K, so nearly every query walks the
// whole cloud; one wave per query re-reading the cloud through the caches
// then moves N x 12 bytes per query from L2 (4096 points, 16384 queries:
// 805 MB), here once per workgroup.  After the copy no wave waits for
// another: each walks its query and leaves.
constexpr int kBqLdsWaves = 16;
constexpr int64_t kBqLdsMinN = 2048;

__global__ __launch_bounds__(64 * kBqLdsWaves) void ball_query_lds_kernel(const float* __restrict__ xyz,
                                                                          const float* __restrict__ qxyz, int N, int M,
                                                                          int qblocks, float r2, int K,
                                                                          int32_t* __restrict__ nit,
                                                                          int32_t* __restrict__ cnt) {
    extern __shared__ float s_pts[];   // [3][N]: x, then y, then z
    const int64_t b = blockIdx.x / qblocks;
    const int q0 = (int)(blockIdx.x - b * qblocks) * kBqLdsWaves;
    const float* __restrict__ p = xyz + b * (int64_t)N * 3;
    for (int e = threadIdx.x; e < 3 * N; e += 64 * kBqLdsWaves) {
        const int j = e / 3;
        s_pts[(e - 3 * j) * N + j] = p[e];
    }
    __syncthreads();
    const int qi = q0 + (int)(threadIdx.x >> 6);
    if (qi >= M) return;   // whole waves leave; no barrier follows
    const int lane = threadIdx.x & 63;
    const int64_t gq = b * M + qi;
    const float* sx = s_pts;
    const float* sy = s_pts + N;
    const float* sz = s_pts + 2 * N;
    auto pt = [&](int j, float& x, float& y, float& z) {
        x = sx[j];
        y = sy[j];
        z = sz[j];
    };
    const int n = bq_walk(pt, N, qxyz[gq * 3 + 0], qxyz[gq * 3 + 1], qxyz[gq * 3 + 2], r2, K, nit + gq * K, lane);
    if (cnt && lane == 0) cnt[gq] = n;
}

// ---------------------------------------------------------------------------
// Grid form for large clouds.
//
// The index-order walk above costs up to N tests per query when a ball holds
// fewer than K points (sparse regions of a LiDAR sweep, whose points come in
// no spatial order).  The grid form bins each cloud into cubic cells of edge
// h >= r (1 + 2^-12), so every point that can pass the test d < fl32(r r)
// lies in the 3 x 3 x 3 cells around the query's cell; a wave tests those
// points in any order and records each hit as a bit of an LDS bitmap over
// the point indices; the first K set bits, read in index order, are the
// first K hits of the walk, bit for bit.
//  * fp32 distances: the computed d is at least D^2 (1 - 4u) and
//    fl32(r r) <= r^2 (1 + u), so a hit has D < r (1 + 3u) < h;
//  * cell coordinates floor((x - min) / h) are computed in fp64 from the
//    fp32 coordinates (the difference is exact), so two points closer than
//    h along an axis are at most one cell apart;
//  * at most 8192 cells per cloud (h grows with the cloud's extent).
// Per call: one workgroup per cloud builds the grid (box, cell shape,
// counts, offsets, cell-grouped copies of the points with their indices),
// then one wave per query searches.
// ---------------------------------------------------------------------------

constexpr int kGridCells = 8192;        // cells per cloud at most (the histogram lives in LDS)
constexpr int kGridQWaves = 4;
constexpr int64_t kBqGridMinN = 8192;   // the grid form runs from this many points

struct GridInfo {
    double mn[3];
    double inv_h;
    int g[3];
    float radius;   // the radius the cells were sized for: they serve queries up to it
};

struct GridWs {
    GridInfo* info;      // [B]
    int32_t* start;      // [B][kGridCells + 1]: exclusive offsets of the cells
    float4* sorted;      // [B][N]: x, y, z, index bits, grouped by cell
};

__device__ __forceinline__ int grid_coord(float x, double mn, double inv_h) {
    const double t = floor(((double)x - mn) * inv_h);
    return (int)fmin(fmax(t, -4.0), 1.0e9);   // far outside: any value below -1 or above g stays clear of the grid
}

__device__ __forceinline__ int grid_cell(const GridInfo& gi, float x, float y, float z) {
    const int cx = min(max(grid_coord(x, gi.mn[0], gi.inv_h), 0), gi.g[0] - 1);
    const int cy = min(max(grid_coord(y, gi.mn[1], gi.inv_h), 0), gi.g[1] - 1);
    const int cz = min(max(grid_coord(z, gi.mn[2], gi.inv_h), 0), gi.g[2] - 1);
    return (cz * gi.g[1] + cy) * gi.g[0] + cx;
}

// One workgroup per cloud: bounding box, cell shape, histogram of the cells
// in LDS, exclusive offsets (written out for the queries), then every point
// copied with its index into its cell's range (order inside a cell is free:
// the queries collect hits in an index bitmap).
__global__ __launch_bounds__(1024) void grid_build_kernel(const float* __restrict__ xyz, int N, float radius,
                                                          GridWs w) {
    const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const float* __restrict__ p = xyz + (int64_t)b * N * 3;
    __shared__ int s_hist[kGridCells + 1];
    __shared__ float s_lo[16][3], s_hi[16][3];
    __shared__ int s_wsum[16];
    __shared__ GridInfo s_gi;
    float lo[3] = {__builtin_huge_valf(), __builtin_huge_valf(), __builtin_huge_valf()};
    float hi[3] = {-__builtin_huge_valf(), -__builtin_huge_valf(), -__builtin_huge_valf()};
    for (int j = tid; j < N; j += 1024)
#pragma unroll
        for (int d = 0; d < 3; ++d) {
            lo[d] = fminf(lo[d], p[3 * j + d]);
            hi[d] = fmaxf(hi[d], p[3 * j + d]);
        }
#pragma unroll
    for (int d = 0; d < 3; ++d)
        for (int o = 32; o > 0; o >>= 1) {
            lo[d] = fminf(lo[d], __shfl_xor(lo[d], o));
            hi[d] = fmaxf(hi[d], __shfl_xor(hi[d], o));
        }
    if (lane == 0)
#pragma unroll
        for (int d = 0; d < 3; ++d) {
            s_lo[wave][d] = lo[d];
            s_hi[wave][d] = hi[d];
        }
    for (int c = tid; c <= kGridCells; c += 1024) s_hist[c] = 0;
    __syncthreads();
    if (tid == 0) {
        double mn[3], e[3];
        for (int d = 0; d < 3; ++d) {
            float a = s_lo[0][d], z = s_hi[0][d];
            for (int v = 1; v < 16; ++v) {
                a = fminf(a, s_lo[v][d]);
                z = fmaxf(z, s_hi[v][d]);
            }
            mn[d] = a;
            e[d] = (double)z - (double)a;
        }
        // cell edge at least r (1 + 2^-12), widened until the cells fit;
        // an edge of a twentieth of the widest extent always fits (20^3
        // cells).  Non-finite coordinates (undefined input) put every point
        // in one cell, so all accesses stay in range.
        const double emax = fmax(e[0], fmax(e[1], e[2]));
        double h = (double)radius * (1.0 + 1.0 / 4096.0);
        if (!(emax < 1.0e300)) {
            e[0] = e[1] = e[2] = 0.0;
        } else {
            auto cells = [&](double hh) {
                return (floor(e[0] / hh) + 1.0) * (floor(e[1] / hh) + 1.0) * (floor(e[2] / hh) + 1.0);
            };
            for (int it = 0; it < 64 && cells(h) > (double)kGridCells; ++it) h *= 1.25;
            if (cells(h) > (double)kGridCells) h = fmax(h, emax / 19.0);
        }
        GridInfo gi;
        for (int d = 0; d < 3; ++d) {
            gi.mn[d] = mn[d];
            gi.g[d] = (int)(floor(e[d] / h) + 1.0);
        }
        gi.inv_h = 1.0 / h;
        gi.radius = radius;
        s_gi = gi;
        w.info[b] = gi;
    }
    __syncthreads();
    const GridInfo gi = s_gi;
    const int ncells = gi.g[0] * gi.g[1] * gi.g[2];
    for (int j = tid; j < N; j += 1024) atomicAdd(&s_hist[grid_cell(gi, p[3 * j], p[3 * j + 1], p[3 * j + 2])], 1);
    __syncthreads();
    // exclusive scan of ncells entries: thread t takes a contiguous run
    const int per = (ncells + 1023) / 1024;
    const int c0 = min(tid * per, ncells), c1 = min(c0 + per, ncells);
    int sum = 0;
    for (int c = c0; c < c1; ++c) sum += s_hist[c];
    int incl = sum;
    for (int o = 1; o < 64; o <<= 1) {
        const int t = __shfl_up(incl, o);
        incl += lane >= o ? t : 0;
    }
    if (lane == 63) s_wsum[wave] = incl;
    __syncthreads();
    int off = incl - sum;
    for (int v = 0; v < wave; ++v) off += s_wsum[v];
    int32_t* st = w.start + (int64_t)b * (kGridCells + 1);
    __syncthreads();   // every thread has read the counts it scans
    for (int c = c0; c < c1; ++c) {
        const int k = s_hist[c];
        s_hist[c] = off;
        st[c] = off;
        off += k;
    }
    if (tid == 0) st[ncells] = N;
    __syncthreads();
    float4* out = w.sorted + (int64_t)b * N;
    for (int j = tid; j < N; j += 1024) {
        const float x = p[3 * j], y = p[3 * j + 1], z = p[3 * j + 2];
        const int slot = atomicAdd(&s_hist[grid_cell(gi, x, y, z)], 1);
        out[slot] = make_float4(x, y, z, __int_as_float(j));
    }
}

// A query whose 27 cells hold more than `walk_above` points sits in a dense
// region, where the index-order walk finds its K hits early: it walks
// instead (same result).
__global__ __launch_bounds__(64 * kGridQWaves) void grid_query_kernel(const float* __restrict__ xyz,
                                                                      const float* __restrict__ qxyz, int64_t BM,
                                                                      int N, int M, float radius, float r2, int K,
                                                                      int walk_above, GridWs w,
                                                                      int32_t* __restrict__ nit,
                                                                      int32_t* __restrict__ cnt) {
    extern __shared__ uint32_t s_bits[];
    const int words = (N + 31) >> 5;
    const int wpl = (words + 63) >> 6;                   // bitmap words per lane
    const int64_t gq = (int64_t)blockIdx.x * kGridQWaves + (threadIdx.x >> 6);
    if (gq >= BM) return;   // whole wave leaves; no barriers below
    const int lane = threadIdx.x & 63;
    uint32_t* bits = s_bits + (threadIdx.x >> 6) * (wpl * 64);
    const int64_t b = gq / M;
    const float qx = qxyz[gq * 3 + 0], qy = qxyz[gq * 3 + 1], qz = qxyz[gq * 3 + 2];
    const GridInfo gi = w.info[b];
    const int32_t* __restrict__ st = w.start + b * (kGridCells + 1);
    const float4* __restrict__ pts = w.sorted + b * N;

    const int cx = grid_coord(qx, gi.mn[0], gi.inv_h);
    const int cy = grid_coord(qy, gi.mn[1], gi.inv_h);
    const int cz = grid_coord(qz, gi.mn[2], gi.inv_h);
    const int x0 = max(cx - 1, 0), x1 = min(cx + 1, gi.g[0] - 1);
    const int y0 = max(cy - 1, 0), y1 = min(cy + 1, gi.g[1] - 1);
    const int z0 = max(cz - 1, 0), z1 = min(cz + 1, gi.g[2] - 1);
    // candidates in the (up to) nine rows of cells, lane t < 9 one row:
    // cells x0 .. x1 of a row are consecutive in the sorted copy, so row t
    // is the range [rs, rs + rn); rp = the rows' inclusive prefix counts
    int rs = 0, rn = 0;
    if (x0 <= x1 && lane < 9) {
        const int y = y0 + lane % 3, z = z0 + lane / 3;
        if (y <= y1 && z <= z1) {
            const int row = (z * gi.g[1] + y) * gi.g[0];
            rs = st[row + x0];
            rn = st[row + x1 + 1] - rs;
        }
    }
    int rp = rn;
    for (int o = 1; o < 16; o <<= 1) {
        const int t = __shfl_up(rp, o);
        rp += lane >= o ? t : 0;
    }
    const int cand = __shfl(rp, 8);
    // a radius above the one the cells were sized for (a grid built apart,
    // mesorasi_ball_query_grid) walks as well: same result
    if (cand > walk_above || !(radius <= gi.radius)) {
        const float* __restrict__ p = xyz + b * (int64_t)N * 3;
        auto pt = [&](int j, float& x, float& y, float& z) {
            x = p[3 * j + 0];
            y = p[3 * j + 1];
            z = p[3 * j + 2];
        };
        const int n = bq_walk(pt, N, qx, qy, qz, r2, K, nit + gq * K, lane);
        if (cnt && lane == 0) cnt[gq] = n;
        return;
    }

    for (int i = 0; i < wpl; ++i) bits[lane * wpl + i] = 0u;
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    // every candidate of the nine rows at once, 64 per pass: candidate c
    // lies in the row whose prefix range holds it (all nine rows' loads in
    // flight together instead of one row after another)
    int rend[9], rdelta[9];
#pragma unroll
    for (int t = 0; t < 9; ++t) {
        rend[t] = __builtin_amdgcn_readlane(rp, t);
        rdelta[t] = __builtin_amdgcn_readlane(rs, t) - (rend[t] - __builtin_amdgcn_readlane(rn, t));
    }
    for (int c0 = 0; c0 < cand; c0 += 64) {
        const int c = c0 + lane;
        bool hit = false;
        int j = 0;
        if (c < cand) {
            int i = c + rdelta[8];
#pragma unroll
            for (int t = 7; t >= 0; --t) i = c < rend[t] ? c + rdelta[t] : i;
            const float4 pt = pts[i];
            j = __float_as_int(pt.w);
            hit = dist3(pt.x, pt.y, pt.z, qx, qy, qz) < r2;
        }
        if (hit) atomicOr(bits + (j >> 5), 1u << (j & 31));
    }
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");

    // the first K set bits in index order: lane l owns words [l wpl, (l+1) wpl)
    int pc = 0;
    for (int i = 0; i < wpl; ++i) pc += __builtin_popcount(bits[lane * wpl + i]);
    int incl = pc;
    for (int o = 1; o < 64; o <<= 1) {
        const int t = __shfl_up(incl, o);
        incl += lane >= o ? t : 0;
    }
    const int total = __shfl(incl, 63);
    int rank = incl - pc;
    int32_t* __restrict__ out = nit + gq * K;
    int lowest = 0x7fffffff;
    for (int i = 0; i < wpl && rank < K; ++i) {
        uint32_t m = bits[lane * wpl + i];
        while (m && rank < K) {
            const int j = ((lane * wpl + i) << 5) + __builtin_ctz(m);
            m &= m - 1u;
            lowest = min(lowest, j);
            out[rank++] = j;
        }
    }
    // the first hit: the lowest index of the lowest lane holding one
    int first = lowest;
    for (int o = 32; o > 0; o >>= 1) first = min(first, __shfl_xor(first, o));
    const int n = min(total, K);
    const int pad = n > 0 ? first : 0;
    for (int k = n + lane; k < K; k += 64) out[k] = pad;
    if (cnt && lane == 0) cnt[gq] = n;
}

static size_t grid_ws_bytes(int64_t B, int64_t N) {
    if (B <= 0 || N <= 0) return 0;
    auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
    return al(B * sizeof(GridInfo)) + al((size_t)B * (kGridCells + 1) * 4) + al((size_t)B * N * 16);
}

static size_t bq_ws_bytes(int64_t B, int64_t N) { return N < kBqGridMinN ? 0 : grid_ws_bytes(B, N); }

static GridWs bq_ws_layout(void* ws, int64_t B, int64_t N) {
    (void)N;
    auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
    char* p = static_cast<char*>(ws);
    GridWs w;
    w.info = reinterpret_cast<GridInfo*>(p);
    p += al(B * sizeof(GridInfo));
    w.start = reinterpret_cast<int32_t*>(p);
    p += al((size_t)B * (kGridCells + 1) * 4);
    w.sorted = reinterpret_cast<float4*>(p);
    return w;
}

static int launch_grid_build(const float* xyz, int64_t B, int64_t N, float radius, const GridWs& w, hipStream_t s,
                             const char* who) {
    MESO_REQUIRE(B <= 0x7fffffff, MESORASI_EUNSUPPORTED, "%s: B too large", who);
    grid_build_kernel<<<dim3((unsigned)B), dim3(1024), 0, s>>>(xyz, (int)N, radius, w);
    return after_launch(who);
}

static int launch_grid_query(const float* xyz, const float* qxyz, int64_t B, int64_t N, int64_t M, float radius,
                             int32_t K, int32_t* nit, int32_t* cnt, const GridWs& w, hipStream_t s, const char* who) {
    const int64_t BM = B * M;
    const int64_t qblocks = ceil_div(BM, kGridQWaves);
    MESO_REQUIRE(qblocks <= 0x7fffffff, MESORASI_EUNSUPPORTED, "%s: too many queries", who);
    const size_t lds = (size_t)kGridQWaves * 64 * ceil_div(ceil_div(N, 32), 64) * 4;
    // walk or grid: a ball of c candidates holds about 0.155 c points
    // (sphere over 27 cubes), so a walk scans about K N / (0.155 c);
    // the two cost the same near c = sqrt(6.45 K N)
    const int walk_above = (int)std::min(std::sqrt(6.45 * (double)K * (double)N), 2.0e9);
    grid_query_kernel<<<dim3((unsigned)qblocks), dim3(64 * kGridQWaves), lds, s>>>(
        xyz, qxyz, BM, (int)N, (int)M, radius, radius * radius, K, walk_above, w, nit, cnt);
    return after_launch(who);
}

// Arguments shared by the ball query entry points.
static int check_bq_args(const char* who, const float* xyz, const float* qxyz, int64_t B, int64_t N, int64_t M,
                         float radius, int32_t K, const int32_t* nit) {
    MESO_REQUIRE(B >= 0 && N >= 0 && M >= 0, MESORASI_EINVAL, "%s: negative size", who);
    MESO_REQUIRE(K >= 1, MESORASI_EINVAL, "%s: K = %d < 1", who, K);
    MESO_REQUIRE(radius > 0.0f && radius <= 3.0e38f, MESORASI_EINVAL, "%s: radius must be finite and > 0", who);
    MESO_REQUIRE(K <= MESORASI_MAX_K_BALL, MESORASI_EUNSUPPORTED, "%s: K = %d > %d", who, K, MESORASI_MAX_K_BALL);
    if (B == 0 || M == 0) return MESORASI_OK;
    MESO_REQUIRE(N >= 1, MESORASI_EINVAL, "%s: N = 0 with M > 0", who);
    MESO_REQUIRE(xyz && qxyz && nit, MESORASI_EINVAL, "%s: NULL xyz, qxyz or nit", who);
    MESO_REQUIRE(N <= 0x7fffffff - 64 * (kBqChunks + 1) && M <= 0x7fffffff, MESORASI_EUNSUPPORTED,
                 "%s: N or M too large", who);
    return MESORASI_OK;
}

}  // namespace meso

using namespace meso;

extern "C" size_t mesorasi_ball_query_workspace(int64_t B, int64_t N, int64_t M) {
    if (B < 0 || N < 0 || M < 0 || N > 0x7fffffff - 64 * (kBqChunks + 1)) return 0;
    return M > 0 ? bq_ws_bytes(B, N) : 0;
}

extern "C" int mesorasi_ball_query(const float* xyz, const float* qxyz, int64_t B, int64_t N, int64_t M,
                                   float radius, int32_t K, int32_t* nit, int32_t* cnt, void* ws, size_t ws_bytes,
                                   void* stream) {
    const char* who = "mesorasi_ball_query";
    int rc = check_bq_args(who, xyz, qxyz, B, N, M, radius, K, nit);
    if (rc != MESORASI_OK || B == 0 || M == 0) return rc;
    const size_t need = bq_ws_bytes(B, N);
    MESO_REQUIRE(ws_bytes >= need && (need == 0 || ws), MESORASI_EWORKSPACE, "%s: workspace %zu < %zu bytes", who,
                 ws_bytes, need);
    MESO_REQUIRE(need == 0 || aligned(ws, 256), MESORASI_EINVAL, "%s: workspace not 256-byte aligned", who);
    MESO_REQUIRE(need == 0 || N <= MESORASI_MAX_N_FPS, MESORASI_EUNSUPPORTED, "%s: N = %lld > %d", who,
                 (long long)N, MESORASI_MAX_N_FPS);
    const float r2 = radius * radius;
    const int64_t BM = B * M;
    hipStream_t s = as_stream(stream);
    if (need > 0) {
        const GridWs w = bq_ws_layout(ws, B, N);
        rc = launch_grid_build(xyz, B, N, radius, w, s, who);
        if (rc != MESORASI_OK) return rc;
        return launch_grid_query(xyz, qxyz, B, N, M, radius, K, nit, cnt, w, s, who);
    }
    if (N >= kBqLdsMinN) {
        // below kBqGridMinN points: 3 N floats of LDS, at most 96 KB
        const int64_t qb = ceil_div(M, kBqLdsWaves);
        MESO_REQUIRE(B * qb <= 0x7fffffff, MESORASI_EUNSUPPORTED, "%s: too many queries", who);
        ball_query_lds_kernel<<<dim3((unsigned)(B * qb)), dim3(64 * kBqLdsWaves), (size_t)N * 12, s>>>(
            xyz, qxyz, (int)N, (int)M, (int)qb, r2, K, nit, cnt);
        return after_launch(who);
    }
    const int64_t blocks = ceil_div(BM, kBqWaves);
    MESO_REQUIRE(blocks <= 0x7fffffff, MESORASI_EUNSUPPORTED, "%s: too many queries", who);
    ball_query_kernel<<<dim3((unsigned)blocks), dim3(64 * kBqWaves), 0, s>>>(xyz, qxyz, BM, (int)N, (int)M, r2, K,
                                                                            nit, cnt);
    return after_launch(who);
}

extern "C" size_t mesorasi_ball_query_grid_workspace(int64_t B, int64_t N) {
    if (B < 0 || N < 0 || N > MESORASI_MAX_N_FPS) return 0;
    return grid_ws_bytes(B, N);
}

extern "C" int mesorasi_ball_query_grid_build(const float* xyz, int64_t B, int64_t N, float radius, void* ws,
                                              size_t ws_bytes, void* stream) {
    const char* who = "mesorasi_ball_query_grid_build";
    MESO_REQUIRE(B >= 0 && N >= 0, MESORASI_EINVAL, "%s: negative size", who);
    MESO_REQUIRE(radius > 0.0f && radius <= 3.0e38f, MESORASI_EINVAL, "%s: radius must be finite and > 0", who);
    MESO_REQUIRE(N <= MESORASI_MAX_N_FPS, MESORASI_EUNSUPPORTED, "%s: N = %lld > %d", who, (long long)N,
                 MESORASI_MAX_N_FPS);
    if (B == 0 || N == 0) return MESORASI_OK;
    MESO_REQUIRE(xyz, MESORASI_EINVAL, "%s: NULL xyz", who);
    const size_t need = grid_ws_bytes(B, N);
    MESO_REQUIRE(ws && ws_bytes >= need, MESORASI_EWORKSPACE, "%s: workspace %zu < %zu bytes", who, ws_bytes, need);
    MESO_REQUIRE(aligned(ws, 256), MESORASI_EINVAL, "%s: workspace not 256-byte aligned", who);
    return launch_grid_build(xyz, B, N, radius, bq_ws_layout(ws, B, N), as_stream(stream), who);
}

extern "C" int mesorasi_ball_query_grid(const float* xyz, const float* qxyz, int64_t B, int64_t N, int64_t M,
                                        float radius, int32_t K, int32_t* nit, int32_t* cnt, const void* ws,
                                        size_t ws_bytes, void* stream) {
    const char* who = "mesorasi_ball_query_grid";
    int rc = check_bq_args(who, xyz, qxyz, B, N, M, radius, K, nit);
    if (rc != MESORASI_OK || B == 0 || M == 0) return rc;
    MESO_REQUIRE(N <= MESORASI_MAX_N_FPS, MESORASI_EUNSUPPORTED, "%s: N = %lld > %d", who, (long long)N,
                 MESORASI_MAX_N_FPS);
    const size_t need = grid_ws_bytes(B, N);
    MESO_REQUIRE(ws && ws_bytes >= need, MESORASI_EWORKSPACE, "%s: workspace %zu < %zu bytes", who, ws_bytes, need);
    MESO_REQUIRE(aligned(ws, 256), MESORASI_EINVAL, "%s: workspace not 256-byte aligned", who);
    return launch_grid_query(xyz, qxyz, B, N, M, radius, K, nit, cnt, bq_ws_layout(const_cast<void*>(ws), B, N),
                             as_stream(stream), who);
}

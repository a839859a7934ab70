// Register-resident shared MLP for narrow fp32 layers on many rows, gfx950.
//
// The per-point MLP F (Sec. 4: with delayed aggregation it runs once per
// input point) on layers of at most 128 channels, e.g. the last feature
// propagation level and the per-point head of the segmentation network
// (65536 rows), where a layer-by-layer GEMM writes and re-reads every
// intermediate activation and stages it through LDS.
//
// Each wave pushes 32-row tiles through every layer on its own.  The
// product is taken transposed, Y^T = W X^T, on v_mfma_f32_32x32x2_f32: the
// weights are the A operand (32 output channels x 2 k) and the activations
// the B operand (2 k x 32 rows), so a lane's 16 accumulators of a 32-channel
// block hold 16 output channels of ONE row, its lane % 32 (channel 8(r/4) +
// 4(lane/32) + r%4 of register r).  An MFMA sums over whatever k order its
// two operands share, so the next layer takes its k steps in exactly that
// register order: step (j, r) is the k pair {32j + 8(r/4) + r%4, +4}, lane
// half h supplying its own accumulator r of block j.  The activations never
// leave registers between layers: no LDS round trip, no barrier, no
// transpose.  The weights, permuted once per workgroup into each layer's k
// order, are the only LDS data: a workgroup is persistent, loads every
// layer's weights and biases once, and its eight waves then stream tiles.
// The first layer reads its rows straight from memory, the two lanes of a
// row taking alternate 4-channel chunks.
#include <algorithm>

#include "common.h"
#include "mlp_internal.h"

namespace meso {

namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kRrWaves = 8;          // waves per workgroup (two per SIMD)
constexpr int kRrMaxWidth = 128;     // widest layer input or output
constexpr int kRrMaxSteps = 64;      // k steps of a layer (128 inputs / 2)
constexpr int kRrMaxLds = 160 * 1024;

struct RrArgs {
    const float* x0;
    int64_t ld0;
    const float* x1;
    int64_t ld1;
    int c0, c1;
    int64_t rows;
    int64_t tiles;
    int n_layers;
    int dims[MESORASI_MAX_LAYERS + 1];
    const float* W[MESORASI_MAX_LAYERS];
    const float* bias[MESORASI_MAX_LAYERS];
    int woff[MESORASI_MAX_LAYERS];   // float offset of layer l's permuted weights in LDS
    int boff[MESORASI_MAX_LAYERS];   // float offset of its padded bias
    int lds_floats;
    // weights staged in phases when all layers do not fit at once: phase p
    // holds layers phase_first[p] .. phase_first[p + 1] - 1 (offsets above
    // relative to the phase); then every wave holds at most one tile
    int nphase;
    int phase_first[MESORASI_MAX_LAYERS + 1];
    uint32_t relu_mask;
    float* y;
    int64_t ldy;
    int k0h;     // layer-0 k values per lane half (a multiple of 16, at most 64)
    int vec0;    // layer-0 rows read as aligned float4 (one source, C0 % 4 == 0)
    int vecy;    // output rows stored as aligned float4
    // interpolated first-layer rows (instead of [x0 | x1]): row r = b Nd + i
    // is phi(sum_k u_k g[b, nn[r, k]] + add[r]) over the first dims[0]
    // channels, u_k the normalised inverse squared distances
    int interp;
    RrInterp ip;
};

__host__ __device__ inline int rr_blocks(int n) { return (n + 31) / 32; }
// k steps of layer l: 16 per 32-channel input block; the first layer's
// half-rows are padded to whole blocks of 16 steps too (k0h = 16 nj)
__host__ __device__ inline int rr_steps(const int* dims, int l, int k0h) {
    return l == 0 ? k0h : 16 * rr_blocks(dims[l]);
}

// The input channel that lane half h supplies at k step s of layer l.
__device__ __forceinline__ int rr_k(int l, int s, int h) {
    // first layer: the two lanes of a row take alternate 4-channel chunks,
    // so a row's 128-byte line is read whole by four consecutive loads
    if (l == 0) return 8 * (s >> 2) + 4 * h + (s & 3);
    const int j = s >> 4, r = s & 15;
    return 32 * j + 8 * (r >> 2) + (r & 3) + 4 * h;
}

// One layer's products: NJ input blocks of 16 k steps, NOB output blocks,
// the output blocks' accumulation chains interleaved step by step.
template <int NJ, int NOB>
__device__ __forceinline__ void rr_products(const float4* __restrict__ wl, const float (&act)[kRrMaxSteps],
                                            f32x16 (&acc)[kRrMaxWidth / 32]) {
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[ob][r] = 0.0f;
    float4 w[NOB];
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob) w[ob] = wl[ob * 4 * NJ * 64];
#pragma unroll
    for (int g = 0; g < 4 * NJ; ++g) {
        // the next group's weights are requested before this group's MFMAs
        float4 wn[NOB];
        if (g + 1 < 4 * NJ) {
#pragma unroll
            for (int ob = 0; ob < NOB; ++ob) wn[ob] = wl[(ob * 4 * NJ + g + 1) * 64];
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int ob = 0; ob < NOB; ++ob)
            acc[ob] = __builtin_amdgcn_mfma_f32_32x32x2f32(w[ob].x, act[4 * g + 0], acc[ob], 0, 0, 0);
#pragma unroll
        for (int ob = 0; ob < NOB; ++ob)
            acc[ob] = __builtin_amdgcn_mfma_f32_32x32x2f32(w[ob].y, act[4 * g + 1], acc[ob], 0, 0, 0);
#pragma unroll
        for (int ob = 0; ob < NOB; ++ob)
            acc[ob] = __builtin_amdgcn_mfma_f32_32x32x2f32(w[ob].z, act[4 * g + 2], acc[ob], 0, 0, 0);
#pragma unroll
        for (int ob = 0; ob < NOB; ++ob)
            acc[ob] = __builtin_amdgcn_mfma_f32_32x32x2f32(w[ob].w, act[4 * g + 3], acc[ob], 0, 0, 0);
        // keeps the compiler from hoisting every group's weights at once
        __builtin_amdgcn_sched_barrier(0);
        if (g + 1 < 4 * NJ) {
#pragma unroll
            for (int ob = 0; ob < NOB; ++ob) w[ob] = wn[ob];
        }
    }
}

template <int NJ>
__device__ __forceinline__ void rr_products_nob(int nob, const float4* __restrict__ wl,
                                                const float (&act)[kRrMaxSteps], f32x16 (&acc)[kRrMaxWidth / 32]) {
    switch (nob) {
        case 1: rr_products<NJ, 1>(wl, act, acc); break;
        case 2: rr_products<NJ, 2>(wl, act, acc); break;
        case 3: rr_products<NJ, 3>(wl, act, acc); break;
        default: rr_products<NJ, 4>(wl, act, acc); break;
    }
}

// Eight waves, two per SIMD: while one wave waits on its rows or runs its
// epilogue, the other keeps the SIMD's MFMA pipe busy.  (A four-wave form
// with 512 registers per wave that requested its next tile's rows before
// computing the current one measured 9-18 % slower.)
// PHASED: the weights staged in phases, at most one tile per wave.
template <bool PHASED>
__global__ __launch_bounds__(64 * kRrWaves) __attribute__((amdgpu_waves_per_eu(2, 2)))
void mlp_rr_kernel(RrArgs a) {
    extern __shared__ float4 smem4[];
    float* smem = reinterpret_cast<float*>(smem4);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int hk = lane >> 5;

    float act[kRrMaxSteps];
    // layer-0 input of tile t: this lane's row; step s takes channel
    // 8 (s / 4) + 4 hk + s % 4
    auto load_tile = [&](int64_t t, float (&dst)[kRrMaxSteps]) {
        const int64_t row = t * 32 + (lane & 31);
        const bool rok = row < a.rows;
        // (opaque per tile: the per-element bounds below are cheap to
        // recompute, while hoisting them out of the tile loop would hold
        // some hundred registers for its whole length)
        int kb = 4 * hk;
        asm volatile("" : "+v"(kb));
        if (a.interp) {
            // the interpolation of mesorasi_interpolate3_add, in its fp32
            // operations, then the addition and phi
            const RrInterp& q = a.ip;
            const int64_t r0 = rok ? row : 0;
            const int64_t b = r0 / q.nd;
            const float w0 = 1.0f / fmaxf(q.dist[r0 * 3 + 0], 1e-10f);
            const float w1 = 1.0f / fmaxf(q.dist[r0 * 3 + 1], 1e-10f);
            const float w2 = 1.0f / fmaxf(q.dist[r0 * 3 + 2], 1e-10f);
            const float ws = w0 + w1 + w2;
            const float u0 = w0 / ws, u1 = w1 / ws, u2 = w2 / ws;
            const float* gs = q.g + b * q.ns * q.ldg;
            const float* g0 = gs + (int64_t)q.nit[r0 * 3 + 0] * q.ldg;
            const float* g1 = gs + (int64_t)q.nit[r0 * 3 + 1] * q.ldg;
            const float* g2 = gs + (int64_t)q.nit[r0 * 3 + 2] * q.ldg;
            const float* ad = q.add + r0 * q.lda;
#pragma unroll
            for (int i = 0; i < kRrMaxSteps / 4; ++i) {
                if (4 * i < a.k0h) {
                    const int k = kb + 8 * i;
                    const bool ok = rok && k < a.c0;
                    const int kk = ok ? k : 0;
                    const float4 x0 = *reinterpret_cast<const float4*>(g0 + kk);
                    const float4 x1 = *reinterpret_cast<const float4*>(g1 + kk);
                    const float4 x2 = *reinterpret_cast<const float4*>(g2 + kk);
                    const float4 p = *reinterpret_cast<const float4*>(ad + kk);
                    float v[4] = {u0 * x0.x + u1 * x1.x + u2 * x2.x, u0 * x0.y + u1 * x1.y + u2 * x2.y,
                                  u0 * x0.z + u1 * x1.z + u2 * x2.z, u0 * x0.w + u1 * x1.w + u2 * x2.w};
                    v[0] += p.x;
                    v[1] += p.y;
                    v[2] += p.z;
                    v[3] += p.w;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        if (q.relu) v[e] = v[e] > 0.0f ? v[e] : 0.0f;
                        dst[4 * i + e] = ok ? v[e] : 0.0f;
                    }
                }
            }
        } else if (a.vec0) {
            const float* src = a.x0 + (rok ? row : 0) * a.ld0;
#pragma unroll
            for (int i = 0; i < kRrMaxSteps / 4; ++i) {
                if (4 * i < a.k0h) {
                    const int k = kb + 8 * i;
                    const bool ok = rok && k < a.c0;
                    const float4 v = *reinterpret_cast<const float4*>(src + (ok ? k : 0));
                    dst[4 * i + 0] = ok ? v.x : 0.0f;
                    dst[4 * i + 1] = ok ? v.y : 0.0f;
                    dst[4 * i + 2] = ok ? v.z : 0.0f;
                    dst[4 * i + 3] = ok ? v.w : 0.0f;
                }
            }
        } else {
            // [x0 | x1] element by element from clamped, in-bounds addresses
            const int64_t r0 = rok ? row : 0;
            const float* src0 = a.x0 + r0 * a.ld0;
            const float* src1 = a.c1 > 0 ? a.x1 + r0 * a.ld1 : src0;
#pragma unroll
            for (int i = 0; i < kRrMaxSteps; ++i) {
                if (i < a.k0h) {
                    const int k = kb + 8 * (i >> 2) + (i & 3);
                    const bool in0 = k < a.c0, in1 = !in0 && k < a.c0 + a.c1;
                    const float v = in0 ? src0[k] : (in1 ? src1[k - a.c0] : src0[0]);
                    dst[i] = (rok && (in0 || in1)) ? v : 0.0f;
                }
            }
        }
    };

    // the first tile's rows are requested before the weights are staged,
    // so their HBM round trip overlaps the staging
    const int64_t stride = (int64_t)gridDim.x * kRrWaves;
    // interpolated rows gather the coarse level's rows of their cloud:
    // workgroups are dealt to the 8 XCDs round-robin by id, so (the grid
    // being a multiple of 8 then) renumber them to give each XCD one
    // contiguous range of tiles -- whole clouds -- and keep those gathers in
    // its own L2
    int64_t wg = blockIdx.x;
    if (a.interp && (gridDim.x & 7) == 0) wg = (int64_t)(blockIdx.x & 7) * (gridDim.x >> 3) + (blockIdx.x >> 3);
    const int64_t t0 = wg * kRrWaves + wave;
    if (t0 < a.tiles) load_tile(t0, act);

    // weights: layer l, output block ob, step group g = s / 4, lane, s % 4;
    // thread tid fills float4s tid + 512 u (u < 8: at most 4 blocks x 16
    // groups x 64 lanes), each 4 consecutive k of one weight row; all of a
    // layer's loads are in flight before the first LDS store
    constexpr int kPer = 4 * 16 * 64 / (64 * kRrWaves);
    auto stage = [&](int l0, int l1) {
        for (int l = l0; l < l1; ++l) {
            const int K = a.dims[l], N = a.dims[l + 1];
            const int ng = rr_steps(a.dims, l, a.k0h) / 4;
            const int total = rr_blocks(N) * ng * 64;
            const unsigned inv = (65536u + ng - 1) / ng;   // gg / ng exactly for gg < 64
            const float* __restrict__ W = a.W[l];
            const bool wvec = (K % 4) == 0 && (reinterpret_cast<uintptr_t>(W) & 15) == 0;
            float4 v[kPer];
#pragma unroll
            for (int u = 0; u < kPer; ++u) {
                const int i = tid + 64 * kRrWaves * u;
                const int ln = i & 63, gg = i >> 6;
                const int ob = (int)(((unsigned)gg * inv) >> 16), g = gg - ob * ng;
                const int n = ob * 32 + (ln & 31);
                const int k = rr_k(l, 4 * g, ln >> 5);   // k .. k + 3 are consecutive
                v[u] = make_float4(0.f, 0.f, 0.f, 0.f);
                if (i < total && n < N) {
                    const float* wr = W + (int64_t)n * K;
                    if (wvec && k + 4 <= K) {
                        v[u] = *reinterpret_cast<const float4*>(wr + k);
                    } else {
                        v[u].x = k + 0 < K ? wr[k + 0] : 0.0f;
                        v[u].y = k + 1 < K ? wr[k + 1] : 0.0f;
                        v[u].z = k + 2 < K ? wr[k + 2] : 0.0f;
                        v[u].w = k + 3 < K ? wr[k + 3] : 0.0f;
                    }
                }
            }
            float4* dst = smem4 + (a.woff[l] >> 2);
#pragma unroll
            for (int u = 0; u < kPer; ++u) {
                const int i = tid + 64 * kRrWaves * u;
                if (i < total) dst[i] = v[u];
            }
            const float* __restrict__ bs = a.bias[l];
            for (int e = tid; e < rr_blocks(N) * 32; e += 64 * kRrWaves)
                smem[a.boff[l] + e] = (bs && e < N) ? bs[e] : 0.0f;
        }
    };

    // layer l on this wave's tile (rows row - lane % 32 ..): act in, act
    // out, or the output rows after the last layer
    auto layer = [&](int l, int64_t row, bool rok) {
        const int N = a.dims[l + 1];
        const int nob = rr_blocks(N);
        const int nj = rr_steps(a.dims, l, a.k0h) / 16;
        const float4* __restrict__ wl = smem4 + (a.woff[l] >> 2) + lane;
        f32x16 acc[kRrMaxWidth / 32];
        switch (nj) {
            case 1: rr_products_nob<1>(nob, wl, act, acc); break;
            case 2: rr_products_nob<2>(nob, wl, act, acc); break;
            case 3: rr_products_nob<3>(nob, wl, act, acc); break;
            default: rr_products_nob<4>(nob, wl, act, acc); break;
        }
        const bool relu = (a.relu_mask >> l) & 1u;
        const float* __restrict__ bl = smem + a.boff[l];
        if (l + 1 < a.n_layers) {
            // bias and activation in place: the accumulators become the
            // next layer's B operand in its k order (steps past the
            // layer's blocks are never read)
#pragma unroll
            for (int ob = 0; ob < kRrMaxWidth / 32; ++ob) {
                if (ob < nob) {
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const float4 b4 = *reinterpret_cast<const float4*>(bl + 32 * ob + 8 * q + 4 * hk);
                        const float bq[4] = {b4.x, b4.y, b4.z, b4.w};
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            float v = acc[ob][4 * q + i] + bq[i];
                            if (relu) v = v > 0.0f ? v : 0.0f;
                            act[16 * ob + 4 * q + i] = v;
                        }
                    }
                }
            }
        } else if (rok) {
            float* yr = a.y + row * a.ldy;
#pragma unroll
            for (int ob = 0; ob < kRrMaxWidth / 32; ++ob) {
                if (ob < nob) {
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const int c = 32 * ob + 8 * q + 4 * hk;
                        const float4 b4 = *reinterpret_cast<const float4*>(bl + c);
                        float v[4] = {acc[ob][4 * q + 0] + b4.x, acc[ob][4 * q + 1] + b4.y,
                                      acc[ob][4 * q + 2] + b4.z, acc[ob][4 * q + 3] + b4.w};
                        if (relu) {
#pragma unroll
                            for (int i = 0; i < 4; ++i) v[i] = v[i] > 0.0f ? v[i] : 0.0f;
                        }
                        if (a.vecy && c + 4 <= N) {
                            *reinterpret_cast<float4*>(yr + c) = make_float4(v[0], v[1], v[2], v[3]);
                        } else {
#pragma unroll
                            for (int i = 0; i < 4; ++i)
                                if (c + i < N) yr[c + i] = v[i];
                        }
                    }
                }
            }
        }
    };

    if constexpr (!PHASED) {
        stage(0, a.n_layers);
        __syncthreads();
        for (int64_t t = t0; t < a.tiles; t += stride) {
            const int64_t row = t * 32 + (lane & 31);
            const bool rok = row < a.rows;
            if (t != t0) load_tile(t, act);
            for (int l = 0; l < a.n_layers; ++l) layer(l, row, rok);
        }
    } else {
        // the weights do not fit at once: the layers run in phases, the
        // workgroup restaging the LDS between them, and each wave holds at
        // most one tile (the host guarantees it), whose activations stay in
        // registers across the phases.  Every wave takes every barrier.
        const int64_t row = t0 * 32 + (lane & 31);
        const bool rok = row < a.rows;
        for (int p = 0; p < a.nphase; ++p) {
            if (p > 0) __syncthreads();   // every wave is done with the previous phase's weights
            stage(a.phase_first[p], a.phase_first[p + 1]);
            __syncthreads();
            if (t0 < a.tiles)
                for (int l = a.phase_first[p]; l < a.phase_first[p + 1]; ++l) layer(l, row, rok);
        }
    }
}

struct RrPlan {
    bool ok;
    int k0h;
    int lds_floats;
    int woff[MESORASI_MAX_LAYERS], boff[MESORASI_MAX_LAYERS];
    int nphase;
    int phase_first[MESORASI_MAX_LAYERS + 1];
};

// Layers packed greedily into phases whose permuted weights and biases fit
// the LDS (one phase when they all fit).
RrPlan rr_plan(int n_layers, const int32_t* dims) {
    RrPlan p{};
    p.k0h = (int)(ceil_div(ceil_div(dims[0], 2), 16) * 16);
    if (p.k0h > kRrMaxSteps || n_layers < 1) return p;
    const int cap = kRrMaxLds / (int)sizeof(float);
    int off = 0, most = 0;
    p.nphase = 1;
    p.phase_first[0] = 0;
    for (int l = 0; l < n_layers; ++l) {
        if (dims[l + 1] > kRrMaxWidth || dims[l] > kRrMaxWidth) return p;
        const int nob = rr_blocks(dims[l + 1]);
        const int size = nob * rr_steps(dims, l, p.k0h) * 64 + nob * 32;
        if (size > cap) return p;
        if (off + size > cap) {
            p.phase_first[p.nphase++] = l;
            off = 0;
        }
        p.woff[l] = off;
        p.boff[l] = off + nob * rr_steps(dims, l, p.k0h) * 64;
        off += size;
        most = std::max(most, off);
    }
    p.phase_first[p.nphase] = n_layers;
    p.lds_floats = most;
    p.ok = true;
    return p;
}

int rr_cus() {
    int dev = 0, cus = 256;
    if (hipGetDevice(&dev) == hipSuccess) {
        int v = 0;
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0) cus = v;
    }
    return cus;
}

}  // namespace

// One phase for any row count; several only while every wave holds at most
// one 32-row tile (one persistent workgroup of kRrWaves waves per CU).
bool rr_mlp_supported(int n_layers, const int32_t* dims, int64_t rows) {
    const RrPlan pl = rr_plan(n_layers, dims);
    return pl.ok && (pl.nphase == 1 || ceil_div(rows, 32) <= (int64_t)rr_cus() * kRrWaves);
}

int run_rr_mlp(const float* x0, int c0, int64_t ld0, const float* x1, int c1, int64_t ld1, int64_t rows,
               int n_layers, const int32_t* dims, const void* const* W, const float* const* bias,
               uint32_t relu_mask, float* y, int64_t ld_y, hipStream_t s, const RrInterp* ip) {
    const RrPlan pl = rr_plan(n_layers, dims);
    MESO_REQUIRE(pl.ok, MESORASI_EUNSUPPORTED, "mesorasi_pointwise_mlp: layers too wide for the register MLP");
    if (rows == 0) return MESORASI_OK;
    const int cus = rr_cus();
    MESO_REQUIRE(pl.nphase == 1 || ceil_div(rows, 32) <= (int64_t)cus * kRrWaves, MESORASI_EUNSUPPORTED,
                 "mesorasi_pointwise_mlp: staged register MLP on more than one tile per wave");
    static const hipError_t attr[2] = {
        hipFuncSetAttribute(reinterpret_cast<const void*>(&mlp_rr_kernel<false>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, kRrMaxLds),
        hipFuncSetAttribute(reinterpret_cast<const void*>(&mlp_rr_kernel<true>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, kRrMaxLds)};
    MESO_REQUIRE(attr[0] == hipSuccess && attr[1] == hipSuccess, MESORASI_EHIP,
                 "mesorasi_pointwise_mlp: LDS size attribute: %s",
                 hipGetErrorString(attr[0] != hipSuccess ? attr[0] : attr[1]));
    RrArgs a{};
    a.x0 = x0; a.ld0 = ld0; a.x1 = x1; a.ld1 = ld1; a.c0 = c0; a.c1 = x1 ? c1 : 0;
    a.rows = rows;
    a.tiles = ceil_div(rows, 32);
    a.n_layers = n_layers;
    for (int l = 0; l <= n_layers; ++l) a.dims[l] = dims[l];
    for (int l = 0; l < n_layers; ++l) {
        a.W[l] = static_cast<const float*>(W[l]);
        a.bias[l] = bias ? bias[l] : nullptr;
        a.woff[l] = pl.woff[l];
        a.boff[l] = pl.boff[l];
    }
    a.lds_floats = pl.lds_floats;
    a.nphase = pl.nphase;
    for (int q = 0; q <= pl.nphase; ++q) a.phase_first[q] = pl.phase_first[q];
    a.relu_mask = relu_mask;
    a.y = y;
    a.ldy = ld_y;
    a.k0h = pl.k0h;
    a.vec0 = a.c1 == 0 && c0 % 4 == 0 && ld0 % 4 == 0 && aligned(x0, 16);
    if (ip) {
        a.interp = 1;
        a.ip = *ip;
        a.c0 = dims[0];
        a.c1 = 0;
    }
    a.vecy = ld_y % 4 == 0 && aligned(y, 16);
    // one persistent workgroup per CU (the weights fill most of the LDS);
    // interpolated rows: a multiple of 8 workgroups where that stays within
    // the CUs (the kernel then orders tiles by XCD)
    int64_t grid = std::min<int64_t>(ceil_div(a.tiles, kRrWaves), cus);
    if (a.interp && 8 * ceil_div(grid, 8) <= cus) grid = 8 * ceil_div(grid, 8);
    const size_t lds = (size_t)pl.lds_floats * sizeof(float);
    if (pl.nphase > 1) mlp_rr_kernel<true><<<dim3((unsigned)grid), dim3(64 * kRrWaves), lds, s>>>(a);
    else mlp_rr_kernel<false><<<dim3((unsigned)grid), dim3(64 * kRrWaves), lds, s>>>(a);
    return after_launch("mesorasi_pointwise_mlp (register MLP)");
}

}  // namespace meso

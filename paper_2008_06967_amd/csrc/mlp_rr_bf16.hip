// Register-resident shared MLP for narrow bf16 layers on many rows, gfx950.
//
// The bf16 form of mlp_rr.hip (the per-point MLP F of Sec. 4 on at most
// 128-channel layers, above 32768 rows: the LiDAR backbone's first module,
// the bf16 segmentation network's first module and per-point head).  The
// arithmetic is that of the bf16 layer-by-layer GEMM: inputs and weights
// rounded to bf16, fp32 accumulation, fp32 bias and ReLU, every stored
// activation (the last layer's output included) rounded to bf16.
//
// Each wave pushes 32-row tiles through every layer on its own, the product
// taken transposed (Y^T = W X^T) on v_mfma_f32_32x32x16_bf16: the weights
// are the A operand, the activations the B operand, and lane l supplies 8
// k values of its own row l % 32 per step (k slot 8 (l / 32) + e).  A
// lane's 16 accumulators of a 32-channel block hold output channels 8(r/4)
// + 4(l/32) + r%4 of its row; rounded to bf16 and packed in pairs they are
// exactly the next layer's B operand if that layer takes, at step t of
// input block j, element e of lane half h to be channel
//   32 j + 16 t + 8 (e / 4) + 4 h + e % 4
// (accumulator r = 8 t + e).  So activations stay in registers between
// layers, 4 registers per step of 16 k.  The first layer reads its rows
// from memory, lane half h taking channels 16 s + 8 h + e at step s.  The
// weights, permuted into these k orders, are staged in LDS once per
// persistent workgroup (16 bytes per lane and step: one LDS read per MFMA).
#include <algorithm>

#include "common.h"
#include "mlp_internal.h"

namespace meso {

namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kRbWaves = 8;          // waves per workgroup (two per SIMD)
constexpr int kRbMaxWidth = 128;     // widest layer input or output
constexpr int kRbMaxSteps = 8;       // k steps of 16 (128 inputs)
constexpr int kRbMaxLds = 160 * 1024;

struct RbArgs {
    const float* x0;
    int64_t ld0;
    const float* x1;
    int64_t ld1;
    int c0, c1;
    int64_t rows;
    int64_t tiles;
    int n_layers;
    int dims[MESORASI_MAX_LAYERS + 1];
    const uint16_t* W[MESORASI_MAX_LAYERS];   // bf16 [C_out, C_in]
    const float* bias[MESORASI_MAX_LAYERS];
    int woff[MESORASI_MAX_LAYERS];   // uint4 offset of layer l's permuted weights in LDS
    int boff[MESORASI_MAX_LAYERS];   // float offset of its padded bias
    uint32_t relu_mask;
    void* y;
    int64_t ldy;
    int out_bf16;
    int vec0;    // layer-0 rows read as aligned float4 (one source, C0 % 4 == 0)
    int vecy;    // output rows stored 4 channels at a time
};

__host__ __device__ inline int rb_blocks(int n) { return (n + 31) / 32; }
__host__ __device__ inline int rb_steps(const int* dims, int l) {
    return l == 0 ? (dims[0] + 15) / 16 : 2 * rb_blocks(dims[l]);
}

// The input channel of element e that lane half h supplies at step s of
// layer l.
__device__ __forceinline__ int rb_k(int l, int s, int h, int e) {
    if (l == 0) return 16 * s + 8 * h + e;
    const int j = s >> 1, t = s & 1;
    return 32 * j + 16 * t + 8 * (e >> 2) + 4 * h + (e & 3);
}

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
    return (uint32_t)f32_to_bf16(lo) | ((uint32_t)f32_to_bf16(hi) << 16);
}

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

// One layer's products: NS steps of 16 k, NOB output blocks, the blocks'
// accumulation chains interleaved; the next step's weights are read before
// this step's MFMAs.
template <int NS, int NOB>
__device__ __forceinline__ void rb_products(const uint4* __restrict__ wl, const uint32_t (&act)[4 * kRbMaxSteps],
                                            f32x16 (&acc)[kRbMaxWidth / 32]) {
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[ob][r] = 0.0f;
    uint4 w[NOB];
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob) w[ob] = wl[ob * NS * 64];
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        uint4 wn[NOB];
        if (s + 1 < NS) {
#pragma unroll
            for (int ob = 0; ob < NOB; ++ob) wn[ob] = wl[(ob * NS + s + 1) * 64];
        }
        __builtin_amdgcn_sched_barrier(0);
        const bf16x8 b = as_bf16x8(make_uint4(act[4 * s], act[4 * s + 1], act[4 * s + 2], act[4 * s + 3]));
#pragma unroll
        for (int ob = 0; ob < NOB; ++ob)
            acc[ob] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(w[ob]), b, acc[ob], 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
        if (s + 1 < NS) {
#pragma unroll
            for (int ob = 0; ob < NOB; ++ob) w[ob] = wn[ob];
        }
    }
}

template <int NS>
__device__ __forceinline__ void rb_products_nob(int nob, const uint4* __restrict__ wl,
                                                const uint32_t (&act)[4 * kRbMaxSteps],
                                                f32x16 (&acc)[kRbMaxWidth / 32]) {
    switch (nob) {
        case 1: rb_products<NS, 1>(wl, act, acc); break;
        case 2: rb_products<NS, 2>(wl, act, acc); break;
        case 3: rb_products<NS, 3>(wl, act, acc); break;
        default: rb_products<NS, 4>(wl, act, acc); break;
    }
}

__global__ __launch_bounds__(64 * kRbWaves) __attribute__((amdgpu_waves_per_eu(2, 2)))
void mlp_rr_bf16_kernel(RbArgs a) {
    extern __shared__ uint4 smem16[];
    float* smemf = reinterpret_cast<float*>(smem16);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int hk = lane >> 5;

    uint32_t act[4 * kRbMaxSteps];
    // layer-0 input of tile t: this lane's row, rounded to bf16; step s
    // takes channels 16 s + 8 hk + e
    auto load_tile = [&](int64_t t) {
        const int64_t row = t * 32 + (lane & 31);
        const bool rok = row < a.rows;
        const int ns = rb_steps(a.dims, 0);
        // (opaque per tile: the per-element bounds below are cheap to
        // recompute, while hoisting them out of the tile loop would hold
        // many registers for its whole length)
        int kb = 8 * hk;
        asm volatile("" : "+v"(kb));
        if (a.vec0) {
            const float* src = a.x0 + (rok ? row : 0) * a.ld0;
#pragma unroll
            for (int s = 0; s < kRbMaxSteps; ++s) {
                if (s < ns) {
                    const int k = kb + 16 * s;
                    const bool ok0 = rok && k < a.c0, ok1 = rok && k + 4 < a.c0;
                    const float4 u = *reinterpret_cast<const float4*>(src + (ok0 ? k : 0));
                    const float4 v = *reinterpret_cast<const float4*>(src + (ok1 ? k + 4 : 0));
                    act[4 * s + 0] = ok0 ? pack_bf16(u.x, u.y) : 0u;
                    act[4 * s + 1] = ok0 ? pack_bf16(u.z, u.w) : 0u;
                    act[4 * s + 2] = ok1 ? pack_bf16(v.x, v.y) : 0u;
                    act[4 * s + 3] = ok1 ? pack_bf16(v.z, v.w) : 0u;
                }
            }
        } else {
            // [x0 | x1] element by element from clamped, in-bounds addresses
            const int64_t r0 = rok ? row : 0;
            const float* src0 = a.x0 + r0 * a.ld0;
            const float* src1 = a.c1 > 0 ? a.x1 + r0 * a.ld1 : src0;
#pragma unroll
            for (int s = 0; s < kRbMaxSteps; ++s) {
                if (s < ns) {
                    float v[8];
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const int k = kb + 16 * s + e;
                        const bool in0 = k < a.c0, in1 = !in0 && k < a.c0 + a.c1;
                        const float x = in0 ? src0[k] : (in1 ? src1[k - a.c0] : src0[0]);
                        v[e] = (rok && (in0 || in1)) ? x : 0.0f;
                    }
#pragma unroll
                    for (int e = 0; e < 4; ++e) act[4 * s + e] = pack_bf16(v[2 * e], v[2 * e + 1]);
                }
            }
        }
    };

    const int64_t stride = (int64_t)gridDim.x * kRbWaves;
    const int64_t t0 = (int64_t)blockIdx.x * kRbWaves + wave;
    if (t0 < a.tiles) load_tile(t0);   // overlaps the weight staging

    // weights: layer l, output block ob, step s, lane -> 8 bf16 (16 bytes)
    for (int l = 0; l < a.n_layers; ++l) {
        const int K = a.dims[l], N = a.dims[l + 1];
        const int ns = rb_steps(a.dims, l);
        const int total = rb_blocks(N) * ns * 64;      // at most 4 x 8 x 64
        const uint16_t* __restrict__ W = a.W[l];
        uint4* dst = smem16 + a.woff[l];
        for (int base = 0; base < total; base += 64 * kRbWaves * 4) {
            uint4 v[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int i = base + tid + 64 * kRbWaves * u;
                const int ln = i & 63, gs = i >> 6;
                const int ob = gs / ns, s = gs - ob * ns;
                const int n = ob * 32 + (ln & 31);
                uint16_t h[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int k = rb_k(l, s, ln >> 5, e);
                    h[e] = (i < total && n < N && k < K) ? W[(int64_t)n * K + k] : (uint16_t)0;
                }
                v[u] = make_uint4(h[0] | ((uint32_t)h[1] << 16), h[2] | ((uint32_t)h[3] << 16),
                                  h[4] | ((uint32_t)h[5] << 16), h[6] | ((uint32_t)h[7] << 16));
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int i = base + tid + 64 * kRbWaves * u;
                if (i < total) dst[i] = v[u];
            }
        }
        const float* __restrict__ bs = a.bias[l];
        for (int e = tid; e < rb_blocks(N) * 32; e += 64 * kRbWaves)
            smemf[a.boff[l] + e] = (bs && e < N) ? bs[e] : 0.0f;
    }
    __syncthreads();

    for (int64_t t = t0; t < a.tiles; t += stride) {
        const int64_t row = t * 32 + (lane & 31);
        const bool rok = row < a.rows;
        if (t != t0) load_tile(t);

        for (int l = 0; l < a.n_layers; ++l) {
            const int N = a.dims[l + 1];
            const int nob = rb_blocks(N);
            const uint4* __restrict__ wl = smem16 + a.woff[l] + lane;
            f32x16 acc[kRbMaxWidth / 32];
            switch (rb_steps(a.dims, l)) {
                case 1: rb_products_nob<1>(nob, wl, act, acc); break;
                case 2: rb_products_nob<2>(nob, wl, act, acc); break;
                case 3: rb_products_nob<3>(nob, wl, act, acc); break;
                case 4: rb_products_nob<4>(nob, wl, act, acc); break;
                case 5: rb_products_nob<5>(nob, wl, act, acc); break;
                case 6: rb_products_nob<6>(nob, wl, act, acc); break;
                case 7: rb_products_nob<7>(nob, wl, act, acc); break;
                default: rb_products_nob<8>(nob, wl, act, acc); break;
            }
            const bool relu = (a.relu_mask >> l) & 1u;
            const float* __restrict__ bl = smemf + a.boff[l];
            // bias, activation, bf16 rounding: channels 32 ob + 8 q + 4 hk + i
            // of accumulator r = 4 q + i
            if (l + 1 < a.n_layers) {
#pragma unroll
                for (int ob = 0; ob < kRbMaxWidth / 32; ++ob) {
                    if (ob < nob) {
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            const float4 b4 = *reinterpret_cast<const float4*>(bl + 32 * ob + 8 * q + 4 * hk);
                            float v[4] = {acc[ob][4 * q + 0] + b4.x, acc[ob][4 * q + 1] + b4.y,
                                          acc[ob][4 * q + 2] + b4.z, acc[ob][4 * q + 3] + b4.w};
                            if (relu) {
#pragma unroll
                                for (int i = 0; i < 4; ++i) v[i] = v[i] > 0.0f ? v[i] : 0.0f;
                            }
                            // accumulator r = 4 q + i is element e = r % 8 of
                            // step 2 ob + r / 8: packed word (2 ob + q / 2) * 4 + (r % 8) / 2
                            const int w0 = 4 * (2 * ob + (q >> 1)) + 2 * (q & 1);
                            act[w0] = pack_bf16(v[0], v[1]);
                            act[w0 + 1] = pack_bf16(v[2], v[3]);
                        }
                    }
                }
            } else if (rok) {
#pragma unroll
                for (int ob = 0; ob < kRbMaxWidth / 32; ++ob) {
                    if (ob < nob) {
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            const int c = 32 * ob + 8 * q + 4 * hk;
                            const float4 b4 = *reinterpret_cast<const float4*>(bl + c);
                            float v[4] = {acc[ob][4 * q + 0] + b4.x, acc[ob][4 * q + 1] + b4.y,
                                          acc[ob][4 * q + 2] + b4.z, acc[ob][4 * q + 3] + b4.w};
                            uint16_t h[4];
#pragma unroll
                            for (int i = 0; i < 4; ++i) {
                                if (relu) v[i] = v[i] > 0.0f ? v[i] : 0.0f;
                                h[i] = f32_to_bf16(v[i]);
                            }
                            if (a.out_bf16) {
                                uint16_t* yr = static_cast<uint16_t*>(a.y) + row * a.ldy + c;
                                if (a.vecy && c + 4 <= N) {
                                    *reinterpret_cast<uint2*>(yr) =
                                        make_uint2(h[0] | ((uint32_t)h[1] << 16), h[2] | ((uint32_t)h[3] << 16));
                                } else {
#pragma unroll
                                    for (int i = 0; i < 4; ++i)
                                        if (c + i < N) yr[i] = h[i];
                                }
                            } else {
                                float* yr = static_cast<float*>(a.y) + row * a.ldy + c;
                                const float4 o = make_float4(bf16_to_f32(h[0]), bf16_to_f32(h[1]),
                                                             bf16_to_f32(h[2]), bf16_to_f32(h[3]));
                                if (a.vecy && c + 4 <= N) {
                                    *reinterpret_cast<float4*>(yr) = o;
                                } else {
                                    const float ov[4] = {o.x, o.y, o.z, o.w};
#pragma unroll
                                    for (int i = 0; i < 4; ++i)
                                        if (c + i < N) yr[i] = ov[i];
                                }
                            }
                        }
                    }
                }
            }
        }
    }
}

struct RbPlan {
    bool ok;
    int lds_bytes;
    int woff[MESORASI_MAX_LAYERS], boff[MESORASI_MAX_LAYERS];
};

RbPlan rb_plan(int n_layers, const int32_t* dims) {
    RbPlan p{};
    if (dims[0] > kRbMaxWidth) return p;
    int off = 0;   // bytes
    for (int l = 0; l < n_layers; ++l) {
        if (dims[l + 1] > kRbMaxWidth) return p;
        const int nob = rb_blocks(dims[l + 1]);
        p.woff[l] = off / 16;
        off += nob * rb_steps(dims, l) * 64 * 16;
        p.boff[l] = off / 4;
        off += nob * 32 * 4;
    }
    if (off > kRbMaxLds) return p;
    p.lds_bytes = off;
    p.ok = true;
    return p;
}

}  // namespace

bool rb_mlp_supported(int n_layers, const int32_t* dims) { return rb_plan(n_layers, dims).ok; }

int run_rb_mlp(const float* x0, int c0, int64_t ld0, const float* x1, int c1, int64_t ld1, int64_t rows,
               int n_layers, const int32_t* dims, const void* const* W, const float* const* bias,
               uint32_t relu_mask, int out_dtype, void* y, int64_t ld_y, hipStream_t s) {
    const RbPlan pl = rb_plan(n_layers, dims);
    MESO_REQUIRE(pl.ok, MESORASI_EUNSUPPORTED, "mesorasi_pointwise_mlp: layers too wide for the register MLP");
    if (rows == 0) return MESORASI_OK;
    static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(&mlp_rr_bf16_kernel),
                                                       hipFuncAttributeMaxDynamicSharedMemorySize, kRbMaxLds);
    MESO_REQUIRE(attr == hipSuccess, MESORASI_EHIP, "mesorasi_pointwise_mlp: LDS size attribute: %s",
                 hipGetErrorString(attr));
    RbArgs a{};
    a.x0 = x0; a.ld0 = ld0; a.x1 = x1; a.ld1 = ld1; a.c0 = c0; a.c1 = x1 ? c1 : 0;
    a.rows = rows;
    a.tiles = ceil_div(rows, 32);
    a.n_layers = n_layers;
    for (int l = 0; l <= n_layers; ++l) a.dims[l] = dims[l];
    for (int l = 0; l < n_layers; ++l) {
        a.W[l] = static_cast<const uint16_t*>(W[l]);
        a.bias[l] = bias ? bias[l] : nullptr;
        a.woff[l] = pl.woff[l];
        a.boff[l] = pl.boff[l];
    }
    a.relu_mask = relu_mask;
    a.y = y;
    a.ldy = ld_y;
    a.out_bf16 = out_dtype == MESORASI_BF16;
    a.vec0 = a.c1 == 0 && c0 % 4 == 0 && ld0 % 4 == 0 && aligned(x0, 16);
    a.vecy = ld_y % 4 == 0 && aligned(y, a.out_bf16 ? 8 : 16);
    int dev = 0, cus = 256;
    if (hipGetDevice(&dev) == hipSuccess) {
        int v = 0;
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0) cus = v;
    }
    const int64_t grid = std::min<int64_t>(ceil_div(a.tiles, kRbWaves), cus);
    mlp_rr_bf16_kernel<<<dim3((unsigned)grid), dim3(64 * kRbWaves), (size_t)pl.lds_bytes, s>>>(a);
    return after_launch("mesorasi_pointwise_mlp (bf16 register MLP)");
}

}  // namespace meso

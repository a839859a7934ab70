// Fused multi-layer shared MLP for narrow layers, gfx950.
//
// With delayed aggregation the MLP runs on the N input points, so its layer
// outputs are small enough to stay on chip (Sec. 4.2: layer outputs shrink
// from 8-32 MB to 512 KB-1 MB).  A workgroup keeps one 64-row tile's
// activations in LDS through all layers (k-major, odd stride); only the last
// layer goes to HBM (or is pooled).  Below 32768 rows, where 64-row tiles
// would leave the CUs one workgroup each, the tiles are 32 rows (one MFMA
// row block), so two workgroups share a CU and overlap each other's loads,
// barriers and epilogues (16384 x 67 -> 64 -> 64 -> 128: 25.6 -> 22.6 us;
// 4096 x 131 -> 128 -> 128 -> 128: 38.8 -> 23.2 us).
//
// Weights never pass through LDS.  Within each 16-wide k-slice the MFMA
// steps use a permuted k order -- lane l at step i takes k = 8*(l/32) + i --
// which MFMA allows as long as both operands agree.  Then the 8 B-operands a
// lane needs for one slice and one 32-column block are 8 consecutive floats
// of one row of W ([C_out, C_in] row-major): two 16-byte loads, fetched a
// slice ahead into registers.  A-operands come from the resident LDS tile.
// Each wave owns whole 32-column blocks (both 32-row halves), so every
// weight is fetched once per workgroup and a layer needs no barrier.
// MFMA: v_mfma_f32_32x32x2_f32 (fp32 in, fp32 accumulate).
// Used for fp32 MLPs whose layer inputs are at most 160 wide and whose
// outputs are at most 128 wide; other MLPs run layer by layer (mlp.hip).
// The conventional module's rows can be gathered straight from the inputs
// through the neighbor index table, which makes that module one kernel:
// gather, every layer, max pool.
#include <type_traits>

#include "common.h"
#include "mlp_internal.h"

namespace meso {

namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));

// H 32-row halves per workgroup tile: 64 rows (H = 2), or 32 rows (H = 1)
// when 64-row tiles would leave the CUs with one workgroup each
constexpr int kOutF32 = 0, kOutBf16 = 1, kOutPool = 2;   // last layer: store fp32 / bf16, or pooled max
template <int H>
constexpr int fst() { return 32 * H + 1; }   // k-major activation stride (odd: conflict-free)
constexpr int kMaxIn = 160;    // widest layer input kept in LDS (padded to 16)
constexpr int kMaxOut = 128;   // widest layer output: 4 column blocks, one per wave

struct FusedArgs {
    const float* x0;
    int64_t ld0;
    const float* x1;
    int64_t ld1;
    int c0, c1;
    int64_t rows;
    int64_t ntiles;    // row tiles (gathered inputs: the grid is padded to a multiple of 8)
    int n_layers;
    int dims[MESORASI_MAX_LAYERS + 1];
    const float* W[MESORASI_MAX_LAYERS];
    const float* bias[MESORASI_MAX_LAYERS];
    uint32_t relu_mask;
    void* y;
    int64_t ldy;
    int out_bf16;
    int64_t G;      // pool group (0: store)
    int hsize;      // floats per activation buffer
    // gathered rows (MlpGather), read at point (r / gmk) * gn + gnit[r]:
    // x0 = xyz minus centroid r / gk of gcen, x1 = feat; or, with lq set,
    // ReLU((x0 - lq[r / gk]) + lb1)
    const int32_t* gnit;
    int64_t gmk, gn;
    int gk;
    const float* gcen;
    const float* lq;
    int64_t ldq;
    const float* lb1;
    // aggregated rows (MlpAggregate): x0 = centroid xyz, x1 = max over the
    // aK rows anit[r, :] of the PFT apft [B, aN, apld] minus its row acidx[r];
    // also stored to aout [rows, aldo] when that is not null
    const float* apft;
    int64_t apld, aN, aM;
    const int32_t* anit;
    const int32_t* acidx;
    int aK;
    float* aout;
    int64_t aldo;
};

constexpr int kInPlain = 0, kInGather = 1, kInAgg = 2;   // layer-0 input forms

__host__ __device__ __forceinline__ int pad16(int x) { return (x + 15) & ~15; }

// 8 consecutive weights W[n][k .. k+7] of a row, from in-bounds addresses:
// a row n >= N reads row 0 and columns k >= K read the row's last column.
// Those values are never used as such -- a column n >= N is never stored,
// and k >= K meets the zeroed k padding of the activation tile (finite
// weights times zero) -- so no select touches the loaded values, and the
// loads stay in flight until the MFMAs of the slice that uses them (a
// select right after the loads made the compiler wait for every slice's
// weights as soon as it requested them, exposing an L2 round trip per
// slice).
// VEC (rows 16-byte aligned, K % 8 == 0): two 16-byte loads, a group past
// K read from the row's last full group (such a group is wholly past K:
// its values meet zero activations); otherwise eight element loads from
// clamped addresses.
template <bool VEC>
__device__ __forceinline__ void load_w8(const float* __restrict__ W, int n, int N, int k, int K, float (&v)[8]) {
    const float* row = W + (int64_t)(n < N ? n : 0) * K;
    if constexpr (VEC) {
        const int kk = min(k, K - 8);
        const float4 a = *reinterpret_cast<const float4*>(row + kk);
        const float4 b = *reinterpret_cast<const float4*>(row + kk + 4);
        v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
        v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
    } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = row[min(k + i, K - 1)];
    }
}

// Column blocks of layer l owned by this wave: cb = wave + 4 j; blocks past
// the layer's count repeat a valid block (discarded) so the MFMA chain stays
// unconditional.
// A layer of at most 64 outputs (one or two blocks) is split by rows
// instead: wave w owns block w / 2 for the 32-row half w % 2, so no wave
// repeats another's MFMAs.
template <int CB, int H>
__device__ __forceinline__ bool row_split(const FusedArgs& a, int l) {
    return H == 2 && CB == 1 && a.dims[l + 1] <= 64;
}

template <int CB, int H>
__device__ __forceinline__ void layer_blocks(const FusedArgs& a, int l, int wave, int (&cbs)[CB]) {
    const int ncb = (a.dims[l + 1] + 31) / 32;
    if (row_split<CB, H>(a, l)) {
        cbs[0] = min(wave >> 1, ncb - 1);
        return;
    }
#pragma unroll
    for (int j = 0; j < CB; ++j) cbs[j] = (wave + 4 * j < ncb) ? wave + 4 * j : min(wave, ncb - 1);
}

__device__ __forceinline__ bool w_vec(const float* W, int K) {
    return K % 8 == 0 && ((reinterpret_cast<uintptr_t>(W) & 15) == 0);
}

// This lane's weights of the first k-slice (k = 0 .. 15) of layer l.
template <int CB, int H>
__device__ __forceinline__ void load_first_slice(const FusedArgs& a, int l, int wave, int lane, float (&w)[CB][8]) {
    const int K = a.dims[l], N = a.dims[l + 1];
    const float* __restrict__ W = a.W[l];
    int cbs[CB];
    layer_blocks<CB, H>(a, l, wave, cbs);
    if (w_vec(W, K)) {
#pragma unroll
        for (int j = 0; j < CB; ++j) load_w8<true>(W, cbs[j] * 32 + (lane & 31), N, 8 * (lane >> 5), K, w[j]);
    } else {
#pragma unroll
        for (int j = 0; j < CB; ++j) load_w8<false>(W, cbs[j] * 32 + (lane & 31), N, 8 * (lane >> 5), K, w[j]);
    }
}

// One layer: hin [K][FST] (LDS) x W^T -> CB column blocks of 32 per wave.
// wb[0] holds this layer's first k-slice on entry (requested before the
// input tile or the previous layer's epilogue, so the weights' round trip
// overlaps that work) and the next layer's on return; the bias is requested
// before the k loop for the same reason.
template <int CB, int OUT, int H>
__device__ __forceinline__ void fused_layer(const FusedArgs& a, int l, const float* __restrict__ hin,
                                            float* __restrict__ hout, int64_t row_t, int tid, int lane, int wave,
                                            float (&wb)[2][CB][8]) {
    const int K = a.dims[l], N = a.dims[l + 1];
    const float* __restrict__ W = a.W[l];
    const int ncb = (N + 31) / 32;
    const bool last = l + 1 == a.n_layers;
    const int kh = 8 * (lane >> 5);              // this lane's half of each 16-slice
    const int cl = lane & 31;
    int cbs[CB];
    constexpr int FST = fst<H>(), FBM = 32 * H;
    layer_blocks<CB, H>(a, l, wave, cbs);
    const float* __restrict__ bias = a.bias[l];
    float bvs[CB];
#pragma unroll
    for (int j = 0; j < CB; ++j) {
        const int col = cbs[j] * 32 + cl;
        bvs[j] = (bias && col < N) ? bias[col] : 0.0f;
    }

    f32x16 acc[CB][H];
#pragma unroll
    for (int j = 0; j < CB; ++j)
#pragma unroll
        for (int h = 0; h < H; ++h)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[j][h][r] = 0.0f;

    const float* hrow = hin + kh * FST + cl;
    const bool split = row_split<CB, H>(a, l);
    const int h0 = wave & 1;

    // the k loop, one copy per weight-load form so the compiler knows how
    // many loads are in flight at every MFMA
    auto kloop = [&](auto vec_c) {
        constexpr bool VEC = decltype(vec_c)::value;
        for (int k0 = 0; k0 < K; k0 += 32) {
            // two slices per trip so the double-buffered weights keep static indices
#pragma unroll
            for (int half = 0; half < 2; ++half) {
                const int ks = k0 + 16 * half;
                if (ks >= K) break;
                // the next slice's weights, requested unconditionally (past
                // K the loads are in-bounds and unused): under a condition
                // the compiler could not count the loads in flight and made
                // every MFMA of the following slice wait for these as well
                if (VEC || ks + 16 < K) {
#pragma unroll
                    for (int j = 0; j < CB; ++j) load_w8<VEC>(W, cbs[j] * 32 + cl, N, ks + 16 + kh, K, wb[half ^ 1][j]);
                }
                if (H == 2 && split) {
                    // this wave's 32-row half only
                    float av[8];
#pragma unroll
                    for (int i = 0; i < 8; ++i) av[i] = hrow[(ks + i) * FST + 32 * h0];
                    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                    for (int i = 0; i < 8; ++i)
                        acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[i], wb[half][0][i], acc[0][0], 0, 0, 0);
                    __builtin_amdgcn_sched_barrier(0);
                } else {
                    float av[8][H];
#pragma unroll
                    for (int i = 0; i < 8; ++i)
#pragma unroll
                        for (int h = 0; h < H; ++h) av[i][h] = hrow[(ks + i) * FST + 32 * h];
                    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                    for (int i = 0; i < 8; ++i)
#pragma unroll
                        for (int j = 0; j < CB; ++j)
#pragma unroll
                            for (int h = 0; h < H; ++h)
                                acc[j][h] =
                                    __builtin_amdgcn_mfma_f32_32x32x2f32(av[i][h], wb[half][j][i], acc[j][h], 0, 0, 0);
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
        }
    };
    if (w_vec(W, K)) kloop(std::true_type{});
    else kloop(std::false_type{});

    if (!last) load_first_slice<CB, H>(a, l + 1, wave, lane, wb[0]);

    // epilogue: bias + ReLU, then LDS (next layer's input) or HBM
    const bool relu = (a.relu_mask >> l) & 1u;
    // one 32-row half h of block j from accumulator v
    auto emit = [&](const f32x16& v, int j, int h) {
        const int col = cbs[j] * 32 + cl;
        const bool col_ok = col < N;
        const float bv = bvs[j];
        const int rbase = h * 32 + 4 * (lane >> 5);
        if (!last) {
            if (col_ok) {
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    float t = v[r] + bv;
                    if (relu) t = t > 0.0f ? t : 0.0f;
                    hout[col * FST + rbase + 8 * (r >> 2) + (r & 3)] = t;
                }
            }
        } else if constexpr (OUT == kOutPool) {
            unsigned* yu = static_cast<unsigned*>(a.y);
            const int64_t half0 = row_t + h * 32;   // 32-row half, a multiple of 32
            if (a.G % 32 == 0) {
                // the whole half lies in one group: fold its 32 rows first.
                // ReLU by comparison maps -0 to +0, so every folded value
                // has a non-negative bit pattern (unsigned atomicMax order)
                float m = 0.0f;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const float t = v[r] + bv;
                    m = fmaxf(m, t > 0.0f ? t : 0.0f);
                }
                m = fmaxf(m, __shfl_xor(m, 32));
                if (lane < 32 && col_ok && half0 < a.rows)
                    atomicMax(yu + (half0 / a.G) * a.ldy + col, __float_as_uint(m));
            } else {
                // groups of this lane's rows: one 64-bit division for the
                // half, then small 32-bit quotients (offsets below G + 32)
                const int64_t rl = row_t + rbase;
                const int64_t g0 = rl / a.G;
                const int off0 = (int)(rl - g0 * a.G);
                const int G = (int)a.G;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int dr = 8 * (r >> 2) + (r & 3);
                    float t = v[r] + bv;
                    t = t > 0.0f ? t : 0.0f;   // pooling requires a final ReLU
                    const int64_t grp = g0 + (unsigned)(off0 + dr) / (unsigned)G;
                    if (col_ok && rl + dr < a.rows) atomicMax(yu + grp * a.ldy + col, __float_as_uint(t));
                }
            }
        } else {
            const int64_t row0 = row_t + rbase;
            if constexpr (OUT == kOutBf16) {
                uint16_t* yb = static_cast<uint16_t*>(a.y) + row0 * a.ldy + col;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int dr = 8 * (r >> 2) + (r & 3);
                    float t = v[r] + bv;
                    if (relu) t = t > 0.0f ? t : 0.0f;
                    if (col_ok && row0 + dr < a.rows) yb[dr * a.ldy] = f32_to_bf16(t);
                }
            } else {
                float* yf = static_cast<float*>(a.y) + row0 * a.ldy + col;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int dr = 8 * (r >> 2) + (r & 3);
                    float t = v[r] + bv;
                    if (relu) t = t > 0.0f ? t : 0.0f;
                    if (col_ok && row0 + dr < a.rows) yf[dr * a.ldy] = t;
                }
            }
        }
    };
    if (H == 2 && split) {
        if ((wave >> 1) < ncb) emit(acc[0][0], 0, h0);
    } else {
#pragma unroll
        for (int j = 0; j < CB; ++j) {
            if (wave + 4 * j >= ncb) continue;
#pragma unroll
            for (int h = 0; h < H; ++h) emit(acc[j][h], j, h);
        }
    }
    if (!last) {
        // zero the k-padding rows of the next input so 0 * garbage never appears
        const int Np = pad16(N);
        for (int e = tid; e < (Np - N) * FBM; e += 256) hout[(N + e / FBM) * FST + (e % FBM)] = 0.0f;
    }
    __syncthreads();
}

// One 32-column block per wave (outputs up to 128 wide), or one block and
// row half for layers of at most 64 outputs; two workgroups per CU (with a
// three-workgroup register budget the row-split epilogue spilled).  (Wider
// outputs measured slower than the per-layer GEMMs.)
template <int CB, int IN, int OUT, int H>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2)))
void mlp_fused_f32_kernel(FusedArgs a) {
    constexpr int FBM = 32 * H, FST = fst<H>();
    extern __shared__ float smem[];
    float* H0 = smem;
    float* H1 = smem + a.hsize;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    int64_t tile = blockIdx.x;
    if constexpr (IN != kInPlain) {
        // gathered rows (a cloud's neighbour rows, or the previous module's
        // feature table): workgroups are dealt to the 8 XCDs round-robin by
        // id, so renumber them to give each XCD one contiguous range of row
        // tiles -- whole clouds -- whose gathered rows then stay in that
        // XCD's L2 instead of every XCD fetching every cloud
        const int64_t per = gridDim.x >> 3;
        tile = (int64_t)(blockIdx.x & 7) * per + (blockIdx.x >> 3);
        if (tile >= a.ntiles) return;   // the whole workgroup, before any barrier
    }
    const int64_t row_t = tile * FBM;
    float wb[2][CB][8];
    load_first_slice<CB, H>(a, 0, wave, lane, wb[0]);

    // layer-0 input tile -> H0 (k-major), zero beyond c0 + c1 up to the slice edge
    {
        const int K0 = a.c0 + a.c1, K0p = pad16(K0);
        if constexpr (IN == kInAgg) {
            // the previous module's aggregation, done here (Sec. 5.2: the
            // aggregation unit writes into the feature buffer of the next
            // MLP): thread t takes row r and four channels, keeps their
            // running max over the row's neighbors (fmaxf from -inf, exact
            // and order-free), subtracts the centroid's row once, and
            // writes the four values into the k-major tile (and to aout)
            const int C4 = a.c1 >> 2;
            for (int e = tid; e < FBM * C4; e += 256) {
                const int r = e / C4, g4 = e - r * C4;
                const int64_t row = row_t + r;
                float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
                if (row < a.rows) {
                    const int64_t b = row / a.aM;
                    const float* __restrict__ base = a.apft + b * a.aN * a.apld + 4 * g4;
                    const int32_t* __restrict__ nr = a.anit + row * a.aK;
                    const float ninf = -__builtin_huge_valf();
                    float4 m = make_float4(ninf, ninf, ninf, ninf);
                    int k = 0;
                    for (; k + 4 <= a.aK; k += 4) {
                        float4 t[4];
#pragma unroll
                        for (int u = 0; u < 4; ++u) t[u] = *reinterpret_cast<const float4*>(base + (int64_t)nr[k + u] * a.apld);
#pragma unroll
                        for (int u = 0; u < 4; ++u) {
                            m.x = fmaxf(m.x, t[u].x);
                            m.y = fmaxf(m.y, t[u].y);
                            m.z = fmaxf(m.z, t[u].z);
                            m.w = fmaxf(m.w, t[u].w);
                        }
                    }
                    for (; k < a.aK; ++k) {
                        const float4 t = *reinterpret_cast<const float4*>(base + (int64_t)nr[k] * a.apld);
                        m.x = fmaxf(m.x, t.x);
                        m.y = fmaxf(m.y, t.y);
                        m.z = fmaxf(m.z, t.z);
                        m.w = fmaxf(m.w, t.w);
                    }
                    const float4 c = *reinterpret_cast<const float4*>(base + (int64_t)a.acidx[row] * a.apld);
                    v = make_float4(m.x - c.x, m.y - c.y, m.z - c.z, m.w - c.w);
                    if (a.aout) *reinterpret_cast<float4*>(a.aout + row * a.aldo + 4 * g4) = v;
                }
                const int k0 = a.c0 + 4 * g4;
                H0[(k0 + 0) * FST + r] = v.x;
                H0[(k0 + 1) * FST + r] = v.y;
                H0[(k0 + 2) * FST + r] = v.z;
                H0[(k0 + 3) * FST + r] = v.w;
            }
            // the centroid coordinates, and zeros up to the slice edge
            for (int e = tid; e < FBM * (K0p - a.c1); e += 256) {
                const int r = e / (K0p - a.c1), kk = e - r * (K0p - a.c1);
                const int k = kk < a.c0 ? kk : a.c1 + kk;
                const int64_t row = row_t + r;
                H0[k * FST + r] = (kk < a.c0 && row < a.rows) ? a.x0[row * a.ld0 + kk] : 0.0f;
            }
        } else if constexpr (IN == kInGather) {
            // gathered rows: each row's input point and centroid once, then
            // the element loop reads them from LDS
            __shared__ int64_t s_pt[FBM], s_cen[FBM];
            if (tid < FBM) {
                const int64_t row = row_t + tid;
                const bool ok = row < a.rows;
                s_pt[tid] = ok ? (row / a.gmk) * a.gn + a.gnit[row] : 0;
                s_cen[tid] = ok ? row / a.gk : 0;
            }
            __syncthreads();
            for (int e = tid; e < FBM * K0p; e += 256) {
                const int r = e / K0p, k = e - r * K0p;
                float v = 0.0f;
                if (row_t + r < a.rows && k < K0) {
                    const int64_t j = s_pt[r], c = s_cen[r];
                    if (a.lq) {
                        const float h = (a.x0[j * a.ld0 + k] - a.lq[c * a.ldq + k]) + (a.lb1 ? a.lb1[k] : 0.0f);
                        v = h > 0.0f ? h : 0.0f;
                    } else if (k < a.c0) {
                        v = a.x0[j * a.ld0 + k] - a.gcen[c * 3 + k];
                    } else {
                        v = a.x1[j * a.ld1 + (k - a.c0)];
                    }
                }
                H0[k * FST + r] = v;
            }
        } else {
            for (int e = tid; e < FBM * K0p; e += 256) {
                const int r = e / K0p, k = e - r * K0p;
                const int64_t row = row_t + r;
                float v = 0.0f;
                if (row < a.rows) {
                    if (k < a.c0) v = a.x0[row * a.ld0 + k];
                    else if (k < K0) v = a.x1[row * a.ld1 + (k - a.c0)];
                }
                H0[k * FST + r] = v;
            }
        }
    }
    __syncthreads();

    for (int l = 0; l < a.n_layers; ++l) {
        const float* hin = (l & 1) ? H1 : H0;
        float* hout = (l & 1) ? H0 : H1;
        fused_layer<CB, OUT, H>(a, l, hin, hout, row_t, tid, lane, wave, wb);
    }
}

}  // namespace

// 32-row tiles when 64-row ones would give fewer than two workgroups per
// CU (256 CUs)
#ifndef MESO_FUSED_H1_BELOW
#define MESO_FUSED_H1_BELOW (64 * 2 * 256)
#endif
static int fused_halves(int64_t rows) { return rows < MESO_FUSED_H1_BELOW ? 1 : 2; }

bool fused_mlp_supported(int n_layers, const int32_t* dims, int dtype) {
    if (dtype != MESORASI_F32 || n_layers < 2) return false;
    for (int l = 0; l < n_layers; ++l)
        if (pad16(dims[l]) > kMaxIn) return false;
    for (int l = 1; l <= n_layers; ++l)
        if (dims[l] > kMaxOut) return false;
    return true;
}

int run_fused_mlp(const float* x0, int c0, int64_t ld0, const float* x1, int c1, int64_t ld1, int64_t rows,
                  int n_layers, const int32_t* dims, const void* const* W, const float* const* bias,
                  uint32_t relu_mask, int out_dtype, void* y, int64_t ld_y, int64_t pool_group, hipStream_t s,
                  const MlpGather* g) {
    FusedArgs a{};
    a.x0 = x0; a.ld0 = ld0; a.x1 = x1; a.ld1 = ld1; a.c0 = c0; a.c1 = c1;
    if (g) {
        a.gnit = g->nit;
        a.gmk = g->mk;
        a.gn = g->n;
        a.gk = g->k;
        a.gcen = g->cxyz;
        a.lq = g->q;
        a.ldq = g->ldq;
        a.lb1 = g->b1;
    }
    a.rows = rows;
    a.n_layers = n_layers;
    int hmax = 16;
    for (int l = 0; l <= n_layers; ++l) a.dims[l] = dims[l];
    for (int l = 0; l < n_layers; ++l) {
        a.W[l] = static_cast<const float*>(W[l]);
        a.bias[l] = bias ? bias[l] : nullptr;
        hmax = std::max(hmax, pad16(dims[l]));   // every layer input (the last output goes to HBM)
    }
    a.relu_mask = relu_mask;
    a.y = y;
    a.ldy = ld_y;
    a.out_bf16 = out_dtype == MESORASI_BF16;
    a.G = pool_group;
    const int H = fused_halves(rows);
    a.hsize = hmax * (32 * H + 1);
    const size_t lds = sizeof(float) * 2 * (size_t)a.hsize;
    if (pool_group > 0) {
        const int rc = zero_rows_f32(static_cast<float*>(y), rows / pool_group, dims[n_layers], ld_y, s);
        if (rc != MESORASI_OK) return rc;
    }
    // one instantiation per input and output form keeps each launch's code
    // (and its instruction-cache footprint) to the path it runs
    const bool gather = g != nullptr;
    a.ntiles = ceil_div(rows, 32 * H);
    const dim3 grid((unsigned)(gather ? 8 * ceil_div(a.ntiles, 8) : a.ntiles)), block(256);
    auto go = [&](auto h) {
        constexpr int HH = decltype(h)::value;
        if (pool_group > 0) {
            if (gather) mlp_fused_f32_kernel<1, kInGather, kOutPool, HH><<<grid, block, lds, s>>>(a);
            else mlp_fused_f32_kernel<1, kInPlain, kOutPool, HH><<<grid, block, lds, s>>>(a);
        } else if (a.out_bf16) {
            if (gather) mlp_fused_f32_kernel<1, kInGather, kOutBf16, HH><<<grid, block, lds, s>>>(a);
            else mlp_fused_f32_kernel<1, kInPlain, kOutBf16, HH><<<grid, block, lds, s>>>(a);
        } else {
            if (gather) mlp_fused_f32_kernel<1, kInGather, kOutF32, HH><<<grid, block, lds, s>>>(a);
            else mlp_fused_f32_kernel<1, kInPlain, kOutF32, HH><<<grid, block, lds, s>>>(a);
        }
    };
    if (H == 1) go(std::integral_constant<int, 1>{});
    else go(std::integral_constant<int, 2>{});
    return after_launch("mesorasi_pointwise_mlp (fused)");
}

int run_fused_aggregate_mlp(const float* cxyz, const MlpAggregate& ag, int64_t rows, int n_layers,
                            const int32_t* dims, const void* const* W, const float* const* bias, uint32_t relu_mask,
                            float* y, int64_t ld_y, hipStream_t s) {
    FusedArgs a{};
    a.x0 = cxyz; a.ld0 = 3; a.c0 = 3; a.c1 = ag.C;
    a.apft = ag.pft; a.apld = ag.ld_pft; a.aN = ag.n; a.aM = ag.m;
    a.anit = ag.nit; a.acidx = ag.cidx; a.aK = ag.k; a.aout = ag.out; a.aldo = ag.ld_out;
    a.rows = rows;
    a.n_layers = n_layers;
    int hmax = 16;
    for (int l = 0; l <= n_layers; ++l) a.dims[l] = dims[l];
    for (int l = 0; l < n_layers; ++l) {
        a.W[l] = static_cast<const float*>(W[l]);
        a.bias[l] = bias ? bias[l] : nullptr;
        hmax = std::max(hmax, pad16(dims[l]));
    }
    a.relu_mask = relu_mask;
    a.y = y;
    a.ldy = ld_y;
    const int H = fused_halves(rows);
    a.hsize = hmax * (32 * H + 1);
    const size_t lds = sizeof(float) * 2 * (size_t)a.hsize;
    a.ntiles = ceil_div(rows, 32 * H);
    const dim3 grid((unsigned)(8 * ceil_div(a.ntiles, 8))), block(256);
    if (H == 1) mlp_fused_f32_kernel<1, kInAgg, kOutF32, 1><<<grid, block, lds, s>>>(a);
    else mlp_fused_f32_kernel<1, kInAgg, kOutF32, 2><<<grid, block, lds, s>>>(a);
    return after_launch("mesorasi_aggregate_mlp");
}

}  // namespace meso

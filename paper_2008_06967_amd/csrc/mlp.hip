// Shared per-point MLP (feature computation F) on gfx950 MFMA, and the
// conventional aggregate-then-MLP module built on it.
//
// F is a matrix-matrix product because all rows share the weights (Sec. 3.1
// "Feature Computation"); with delayed aggregation it runs on the N input
// points instead of the N_out x K neighbor rows (Sec. 4.1, Eq. (3)).
//
// One launch per layer: Y = phi(X W^T + b) with X = [x0 | x1] (two column
// sources, so the first layer reads xyz and the previous module's features
// without a concatenated copy).  Workgroup tiles of 64 or 128 rows by 64 or
// 128 output channels (chosen per layer to fill the 256 CUs; fp32 tiles of
// 128 rows run with eight waves, and with 256 rows when a layer has a full
// wave of those), each wave owning up to 2 x 2 blocks of 32 x 32; layers
// with too few tiles split K and sum the partials in a fixed order:
//  - fp32: v_mfma_f32_32x32x2_f32 (lane l feeds one A and one B value of
//    the same k); row-major LDS tiles read with 16-byte loads in an MFMA
//    lane k-order (details at gemm_f32_kernel).
//  - bf16: v_mfma_f32_32x32x16_bf16 (lane l feeds 8 consecutive k of row
//    l%32, k offset 8*(l/32)); LDS rows of 32 bf16 padded to 40 so the
//    16-byte reads of a half wave hit distinct banks.
// The accumulator of a 32 x 32 MFMA holds, in lane l and register r, row
// 8*(r/4) + 4*(l/32) + r%4 and column l%32.
// Epilogue: + bias, optional ReLU, optional bf16 rounding, then either a
// store or a pooled column max (pool groups of G rows; values are >= 0
// after ReLU, so the max is an unsigned atomicMax on the float bits, which
// is exact and order independent).
// MLPs on at most 64 rows (the classifier head) take a skinny path of
// 16-column MFMA blocks instead (skinny_f32_kernel); narrow multi-layer fp32
// MLPs run fused in one kernel (mlp_fused.hip).
#include <mutex>

#include "common.h"
#include "mlp_internal.h"

namespace meso {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int BKH = 32;      // bf16 k-slice
constexpr int kPadF = 4;     // fp32 k-major LDS rows: tile width + 4 words
constexpr int kRowH = 32;    // bf16 LDS rows: 32 k (64 bytes, four 16-byte chunks), unpadded

// Chunk c of LDS row r of the bf16 tiles sits at chunk position c ^ s(r):
// the eight (or sixteen) lanes of one 16-byte LDS access phase then touch
// every bank once, both for the tile stores (four lanes per row) and for
// the operand reads (one row per lane, one chunk), with 32 or with 64
// banks of 4 bytes.
__device__ __forceinline__ int bf16_chunk(int r, int c) { return 8 * (c ^ (((r >> 1) + (r >> 3)) & 3)); }
constexpr int kTargetTiles = 256;   // one tile per CU

enum { EPI_F32 = 0, EPI_BF16 = 1, EPI_POOL = 2, EPI_PARTIAL = 3 };

struct GemmArgs {
    const void* x0;
    int64_t ld0;
    const float* x1;
    int64_t ld1;
    int c0, c1;
    int a_bf16;          // x0 holds bf16 bits (intermediate activations of the bf16 path)
    int64_t rows;
    int K, N;
    int kc;              // K range per split (multiple of the k-slice)
    const void* W;       // [N, K]
    const float* bias;   // [N] or null
    int relu;
    int round_bf16;      // round activations to bf16 (bf16 path)
    void* y;
    int64_t ldy;
    int64_t G;           // pool group (EPI_POOL)
    float* part;         // split-K partial sums [splits, rows, N]
    // two-source first layer with a narrow x0 (the xyz columns): the main
    // loop runs over x1 alone against W columns cc .. cc + K - 1 (row stride
    // ldw), and the cc x0 columns are added in the epilogue
    const float* xc;
    int64_t ldc;
    int cc;
    int ldw;
    // pooled output of the MLP's last layer, cleared by the first layer's
    // workgroups (null: nothing to clear)
    float* zy;
    int64_t zrows, zld;
    int zcols;
    // gathered first layer of the conventional module (split form only):
    // row r reads point g = (r / gmk) * gn + gnit[r] of the inputs -- x1
    // row g and, through xc, xyz row g minus centroid row r / gk of gcen
    const int32_t* gnit;
    int64_t gmk, gn;
    int gk;
    const float* gcen;
    // gathered layer of the limited order (lq set, single fast source):
    // input row r is ReLU((x0[g] - lq[r / gk]) + lb1)
    const float* lq;
    int64_t ldq;
    const float* lb1;
};

// Input row of row r of a gathered layer (see GemmArgs::gnit).
__device__ __forceinline__ int64_t gather_row(const GemmArgs& a, int64_t r) {
    return (r / a.gmk) * a.gn + a.gnit[r];
}

// Clears the pooled output from the first layer's kernel, so the last
// layer's atomic maxima start from zero without a separate fill launch
// (kernel order on the stream makes the clear complete first).
__device__ __forceinline__ void clear_pool_target(const GemmArgs& a) {
    if (!a.zy) return;
    const int64_t nb = (int64_t)gridDim.x * gridDim.y * gridDim.z;
    const int64_t bid = blockIdx.x + (int64_t)gridDim.x * (blockIdx.y + (int64_t)gridDim.y * blockIdx.z);
    const int64_t n = a.zrows * a.zcols;
    for (int64_t e = bid * blockDim.x + threadIdx.x; e < n; e += nb * blockDim.x)
        a.zy[(e / a.zcols) * a.zld + e % a.zcols] = 0.0f;
}

// 16 bytes at a 4-byte aligned address: gfx950 global loads accept dword
// alignment, so this is still one 16-byte load.
struct __attribute__((packed, aligned(4))) f32x4u {
    float x, y, z, w;
};

// Element (r, k) of the virtual input [x0 | x1] as float (0 outside).
__device__ __forceinline__ float a_elem(const GemmArgs& a, int64_t r, int k) {
    if (r >= a.rows) return 0.0f;
    if (k < a.c0) {
        if (a.a_bf16) return bf16_to_f32(static_cast<const uint16_t*>(a.x0)[r * a.ld0 + k]);
        return static_cast<const float*>(a.x0)[r * a.ld0 + k];
    }
    k -= a.c0;
    if (k < a.c1) return a.x1[r * a.ld1 + k];
    return 0.0f;
}

// L consecutive input elements (r, k0 .. k0+L-1) as float, L in {4, 8}.
// The fast form always loads from a clamped, in-bounds address and zeroes
// out-of-range values by selection: no divergent branch, so a prefetch can
// stay in flight across the MFMAs that follow it.
template <int L, bool FAST>
__device__ __forceinline__ void load_a(const GemmArgs& a, int64_t r, int k0, float (&v)[L], bool& ok) {
    if constexpr (FAST) {
        // single fp32 source, 16-byte aligned rows, K a multiple of 8; the
        // caller zeroes the values when !ok (at its LDS store)
        ok = r < a.rows && k0 < a.K;
        const int64_t rc = ok ? r : 0;
        const int kc = ok ? k0 : 0;
        const float4* p = reinterpret_cast<const float4*>(static_cast<const float*>(a.x0) + rc * a.ld0 + kc);
#pragma unroll
        for (int h = 0; h < L / 4; ++h) {
            const float4 u = p[h];
            v[4 * h + 0] = u.x;
            v[4 * h + 1] = u.y;
            v[4 * h + 2] = u.z;
            v[4 * h + 3] = u.w;
        }
    } else {
        ok = true;
#pragma unroll
        for (int i = 0; i < L; ++i) v[i] = a_elem(a, r, k0 + i);
    }
}

// L consecutive elements (r, k0 ..) of [x0 | x1] for fp32 sources of any
// widths and alignment: per element the address is selected (clamped to the
// row's first element when past K) and the value zeroed, without branches,
// so the loads stay in flight like the vector ones.
template <int L>
__device__ __forceinline__ void load_a_mixed(const GemmArgs& a, int64_t r, int k0, float (&v)[L], bool& ok) {
    ok = r < a.rows;
    const int64_t rr = ok ? r : 0;
    const float* r0 = static_cast<const float*>(a.x0) + rr * a.ld0;
    const float* r1 = a.x1 ? a.x1 + rr * a.ld1 : r0;
#pragma unroll
    for (int i = 0; i < L; ++i) {
        const int k = k0 + i;
        const bool in0 = k < a.c0;
        const bool in1 = !in0 && k < a.K;
        const float* p = in0 ? r0 + k : (in1 ? r1 + (k - a.c0) : r0);
        const float t = *p;
        v[i] = (in0 || in1) ? t : 0.0f;
    }
}

// L consecutive weights (n, k0 ..) for rows of any length, branch-free.
template <int L>
__device__ __forceinline__ void load_w_mixed(const GemmArgs& a, int n, int k0, float (&v)[L], bool& ok) {
    ok = n < a.N;
    const float* wr = static_cast<const float*>(a.W) + (int64_t)(ok ? n : 0) * a.K;
#pragma unroll
    for (int i = 0; i < L; ++i) {
        const bool in = k0 + i < a.K;
        const float t = *(in ? wr + k0 + i : wr);
        v[i] = in ? t : 0.0f;
    }
}

template <int L, bool FAST>
__device__ __forceinline__ void load_w_f32(const GemmArgs& a, int n, int k0, float (&v)[L], bool& ok) {
    const float* W = static_cast<const float*>(a.W);
    if constexpr (FAST) {
        ok = n < a.N && k0 < a.K;
        const float4* p = reinterpret_cast<const float4*>(W + (int64_t)(ok ? n : 0) * a.K + (ok ? k0 : 0));
#pragma unroll
        for (int h = 0; h < L / 4; ++h) {
            const float4 u = p[h];
            v[4 * h + 0] = u.x;
            v[4 * h + 1] = u.y;
            v[4 * h + 2] = u.z;
            v[4 * h + 3] = u.w;
        }
        return;
    }
    ok = true;
#pragma unroll
    for (int i = 0; i < L; ++i) v[i] = (n < a.N && k0 + i < a.K) ? W[(int64_t)n * a.K + k0 + i] : 0.0f;
}

__device__ __forceinline__ uint4 select_u4(bool ok, uint4 q) {
    return make_uint4(ok ? q.x : 0u, ok ? q.y : 0u, ok ? q.z : 0u, ok ? q.w : 0u);
}

template <bool FAST>
__device__ __forceinline__ uint4 load_w8_bf16(const GemmArgs& a, int n, int k0, bool& ok) {
    const uint16_t* W = static_cast<const uint16_t*>(a.W);
    if (FAST) {
        ok = n < a.N && k0 < a.K;
        return *reinterpret_cast<const uint4*>(W + (int64_t)(ok ? n : 0) * a.K + (ok ? k0 : 0));
    }
    ok = n < a.N;
    const uint16_t* wr = W + (int64_t)(ok ? n : 0) * a.K;
    uint16_t h[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const bool in = k0 + i < a.K;
        const uint16_t t = *(in ? wr + k0 + i : wr);
        h[i] = in ? t : (uint16_t)0;
    }
    uint4 q;
    q.x = h[0] | ((uint32_t)h[1] << 16);
    q.y = h[2] | ((uint32_t)h[3] << 16);
    q.z = h[4] | ((uint32_t)h[5] << 16);
    q.w = h[6] | ((uint32_t)h[7] << 16);
    return q;
}

// Load 8 input elements as bf16 bits (rounding fp32 sources to nearest even).
template <bool FAST>
__device__ __forceinline__ uint4 load_a8_bf16(const GemmArgs& a, int64_t r, int k0, bool& ok) {
    if (a.a_bf16 && FAST) {
        ok = r < a.rows && k0 < a.K;
        return *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(a.x0) + (ok ? r : 0) * a.ld0 +
                                               (ok ? k0 : 0));
    }
    ok = true;
    uint16_t h[8];
    if (a.a_bf16) {
#pragma unroll
        for (int i = 0; i < 8; ++i)
            h[i] = (r < a.rows && k0 + i < a.c0) ? static_cast<const uint16_t*>(a.x0)[r * a.ld0 + k0 + i] : (uint16_t)0;
    } else {
        float v[8];
        bool okv;
        if constexpr (FAST) load_a<8, true>(a, r, k0, v, okv);
        else load_a_mixed<8>(a, r, k0, v, okv);
#pragma unroll
        for (int i = 0; i < 8; ++i) h[i] = f32_to_bf16(okv ? v[i] : 0.0f);
    }
    uint4 q;
    q.x = h[0] | ((uint32_t)h[1] << 16);
    q.y = h[2] | ((uint32_t)h[3] << 16);
    q.z = h[4] | ((uint32_t)h[5] << 16);
    q.w = h[6] | ((uint32_t)h[7] << 16);
    return q;
}

// bias, ReLU and (bf16 path) rounding of one pre-activation value
template <bool ROUND>
__device__ __forceinline__ float activate(const GemmArgs& a, float t, float bias) {
    t += bias;
    if (a.relu) t = t > 0.0f ? t : 0.0f;
    if constexpr (ROUND) t = round_bf16(t);
    return t;
}

// Epilogue of one 32 x 32 accumulator block at (row0, col0).  ROUND: the
// bf16 path rounds every stored activation to bf16.
template <int EPI, bool ROUND>
__device__ __forceinline__ void epilogue(const GemmArgs& a, const f32x16& acc, int64_t row0, int col0, int lane) {
    const int col = col0 + (lane & 31);
    const bool col_ok = col < a.N;
    const int64_t rbase = row0 + 4 * (lane >> 5);
    if constexpr (EPI == EPI_PARTIAL) {
        if (!col_ok) return;
        float* part = a.part + (int64_t)blockIdx.z * a.rows * a.N;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int64_t row = rbase + 8 * (r >> 2) + (r & 3);
            if (row < a.rows) part[row * a.N + col] = acc[r];
        }
        return;
    }
    const float bias = (col_ok && a.bias) ? a.bias[col] : 0.0f;
    float v[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) v[r] = activate<ROUND>(a, acc[r], bias);
    if constexpr (EPI == EPI_POOL) {
        unsigned* yu = static_cast<unsigned*>(a.y);
        if (a.G % 32 == 0) {
            // the whole 32-row block lies in one group (row0 is a multiple of 32)
            if (row0 >= a.rows) return;
            float m = v[0];
#pragma unroll
            for (int r = 1; r < 16; ++r) m = fmaxf(m, v[r]);
            m = fmaxf(m, __shfl_xor(m, 32));
            if (lane < 32 && col_ok) atomicMax(yu + (row0 / a.G) * a.ldy + col, __float_as_uint(m));
            return;
        }
        // this lane's rows rbase + d (d < 32): one 64-bit division, then
        // 32-bit quotients of offsets below G + 32 (the caller keeps G < 2^31)
        const int64_t gb = rbase / a.G;
        const unsigned ob = (unsigned)(rbase - gb * a.G), G = (unsigned)a.G;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int64_t r0 = rbase + 8 * q;  // rows r0 .. r0 + 3 in registers 4q .. 4q+3
            if (!col_ok || r0 >= a.rows) continue;
            const unsigned o = ob + 8 * q;
            const int nr = r0 + 3 < a.rows ? 4 : (int)(a.rows - r0);
            const int64_t g0 = gb + o / G;
            if (gb + (o + nr - 1) / G == g0) {
                float m = v[4 * q];
                for (int i = 1; i < nr; ++i) m = fmaxf(m, v[4 * q + i]);
                atomicMax(yu + g0 * a.ldy + col, __float_as_uint(m));
            } else {
                for (int i = 0; i < nr; ++i)
                    atomicMax(yu + (gb + (o + i) / G) * a.ldy + col, __float_as_uint(v[4 * q + i]));
            }
        }
    } else {
        if (!col_ok) return;
        if (row0 + 32 <= a.rows) {
            // whole block in range: unguarded stores
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int64_t row = rbase + 8 * (r >> 2) + (r & 3);
                if constexpr (EPI == EPI_F32) static_cast<float*>(a.y)[row * a.ldy + col] = v[r];
                else static_cast<uint16_t*>(a.y)[row * a.ldy + col] = f32_to_bf16(v[r]);
            }
            return;
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int64_t row = rbase + 8 * (r >> 2) + (r & 3);
            if (row < a.rows) {
                if constexpr (EPI == EPI_F32) static_cast<float*>(a.y)[row * a.ldy + col] = v[r];
                else static_cast<uint16_t*>(a.y)[row * a.ldy + col] = f32_to_bf16(v[r]);
            }
        }
    }
}

// fp32 MFMA GEMM.  Workgroup tile BM x BN, NW waves in an (NW / 2) x 2 grid
// (four or eight: eight put two waves on each SIMD), each wave TM x TN
// blocks of 32 x 32.  K advances in slices of BK through double-buffered
// row-major LDS tiles (rows of BK words + 4 pad); the next slice is fetched
// into registers while the current one feeds the MFMAs, so one barrier per
// slice suffices.  Inside a slice the k order is permuted to the MFMA lane
// layout: at step kk lane l contributes k = (BK/2)*(l/32) + kk for both
// operands, so each lane's operands of a slice are BK/2 consecutive words
// of one LDS row, read with 16-byte loads (conflict-free: row stride
// BK + 4 words puts 8 consecutive lanes on distinct bank quads).  The
// product is the same sum over k, accumulated in a different order.
//
// SPLIT (first layer [x0 | x1] with x0 at most 4 columns wide and x1
// 16-byte aligned): the k loop reads x1 like a single fast source and the
// weight columns after x0 with unaligned 16-byte loads; the x0 columns and
// their weights are staged in LDS once and added to the accumulators before
// the epilogue (same sum, different order).  A gathered split layer (the
// conventional module's first layer) takes its rows through the neighbor
// index table, so the neighbor feature matrix is never written to memory.
template <int BM, int BN, int BK, int EPI, bool FAST_A, bool FAST_W, bool SPLIT = false, bool LTD = false,
          int NW = 4>
__global__ __launch_bounds__(64 * NW) void gemm_f32_kernel(GemmArgs a) {
    static_assert(!SPLIT || FAST_A, "the split form reads x1 as a fast source");
    static_assert(!LTD || (FAST_A && FAST_W && !SPLIT), "the limited-order gather reads one fast source");
    constexpr int NTHR = 64 * NW;            // waves in a (NW / 2) x 2 grid, WRM x WRN each
    constexpr int WRM = BM / (NW / 2), WRN = BN / 2;
    constexpr int TM = WRM / 32, TN = WRN / 32;
    constexpr int LW = BK + kPadF;           // LDS row stride in words
    constexpr int CPR = BK / 4;              // 16-byte chunks per tile row
    static_assert(WRM % 32 == 0 && WRN % 32 == 0, "whole 32 x 32 MFMA blocks per wave");
    constexpr int QA = BM * CPR / NTHR, QB = BN * CPR / NTHR;   // chunks per thread per slice
    constexpr int HK = BK / 2;               // k per lane per slice
    static_assert(QA >= 1 && QB >= 1 && HK % 4 == 0, "tile shape");
    __shared__ __attribute__((aligned(16))) float As[2][BM * LW];
    __shared__ __attribute__((aligned(16))) float Bs[2][BN * LW];
    __shared__ __attribute__((aligned(16))) float sXc[SPLIT ? BM * 4 : 4];
    __shared__ __attribute__((aligned(16))) float sWc[SPLIT ? BN * 4 : 4];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int64_t row_t = (int64_t)blockIdx.x * BM;
    const int col_t = blockIdx.y * BN;
    const int ldw = SPLIT ? a.ldw : a.K;
    clear_pool_target(a);
    if constexpr (SPLIT) {
        // x0 rows of this tile and the matching weight columns (zero past
        // cc, rows or N); read after the first barrier below
        const float* Wf = static_cast<const float*>(a.W) - a.cc;
        for (int e = tid; e < BM * 4; e += NTHR) {
            const int64_t r = row_t + (e >> 2);
            const int i = e & 3;
            float v = 0.0f;
            if (i < a.cc && r < a.rows) {
                if (a.gnit) v = a.xc[gather_row(a, r) * a.ldc + i] - a.gcen[(r / a.gk) * 3 + i];
                else v = a.xc[r * a.ldc + i];
            }
            sXc[e] = v;
        }
        for (int e = tid; e < BN * 4; e += NTHR) {
            const int n = col_t + (e >> 2);
            const int i = e & 3;
            sWc[e] = (i < a.cc && n < a.N) ? Wf[(int64_t)n * ldw + i] : 0.0f;
        }
    }
    const int k_lo = blockIdx.z * a.kc;
    const int k_hi = min(a.K, k_lo + a.kc);
    // chunk c = tid + NTHR p covers tile row c / CPR, words 4 (c % CPR) .. +3
    const int crow = tid / CPR, ck = 4 * (tid % CPR);
    constexpr int RSTEP = NTHR / CPR;        // tile rows between a thread's chunks

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    // Two register stages alternate, so the global loads of a slice are
    // issued two slices before its LDS store: their latency is covered by
    // two slices of MFMAs.  Fast sources keep one clamped row pointer per
    // chunk; a chunk past K loads column 0 of its row and is zeroed at the
    // store, so every address stays inside the operand.
    float ra0[QA][4], rb0[QB][4], ra1[QA][4], rb1[QB][4];
    bool oka0[QA], okb0[QB], oka1[QA], okb1[QB];
    const float* pa[QA];
    const float* pq[LTD ? QA : 1];
    const float* pb[QB];
    bool rowa[QA], rowb[QB];
#pragma unroll
    for (int p = 0; p < QA; ++p) {
        const int64_t r = row_t + crow + RSTEP * p;
        rowa[p] = r < a.rows;
        int64_t src = rowa[p] ? r : 0;
        if constexpr (SPLIT || LTD) {
            if (a.gnit && rowa[p]) src = gather_row(a, r);
        }
        pa[p] = static_cast<const float*>(a.x0) + src * a.ld0;
        if constexpr (LTD) pq[p] = a.lq + (rowa[p] ? r / a.gk : 0) * a.ldq;
    }
#pragma unroll
    for (int p = 0; p < QB; ++p) {
        const int n = col_t + crow + RSTEP * p;
        rowb[p] = n < a.N;
        pb[p] = static_cast<const float*>(a.W) + (int64_t)(rowb[p] ? n : 0) * ldw;
    }
    auto fetch = [&](float (&ra)[QA][4], bool (&oka)[QA], float (&rb)[QB][4], bool (&okb)[QB], int k0) {
        const bool kin = k0 + ck < a.K;
        const int ko = kin ? k0 + ck : 0;    // columns past K read column 0 of the row
#pragma unroll
        for (int p = 0; p < QA; ++p) {
            if constexpr (LTD) {
                const float4 u = *reinterpret_cast<const float4*>(pa[p] + ko);
                const float4 qv = *reinterpret_cast<const float4*>(pq[p] + ko);
                const float4 bv = a.lb1 ? *reinterpret_cast<const float4*>(a.lb1 + ko) : make_float4(0.f, 0.f, 0.f, 0.f);
                const float h[4] = {(u.x - qv.x) + bv.x, (u.y - qv.y) + bv.y, (u.z - qv.z) + bv.z, (u.w - qv.w) + bv.w};
#pragma unroll
                for (int i = 0; i < 4; ++i) ra[p][i] = h[i] > 0.0f ? h[i] : 0.0f;
                oka[p] = rowa[p] && kin;
            } else if constexpr (FAST_A) {
                const float4 u = *reinterpret_cast<const float4*>(pa[p] + ko);
                ra[p][0] = u.x; ra[p][1] = u.y; ra[p][2] = u.z; ra[p][3] = u.w;
                oka[p] = rowa[p] && kin;
            } else {
                load_a_mixed<4>(a, row_t + crow + RSTEP * p, k0 + ck, ra[p], oka[p]);
            }
        }
#pragma unroll
        for (int p = 0; p < QB; ++p) {
            if constexpr (SPLIT) {
                const f32x4u u = *reinterpret_cast<const f32x4u*>(pb[p] + ko);
                rb[p][0] = u.x; rb[p][1] = u.y; rb[p][2] = u.z; rb[p][3] = u.w;
                okb[p] = rowb[p] && kin;
            } else if constexpr (FAST_W) {
                const float4 u = *reinterpret_cast<const float4*>(pb[p] + ko);
                rb[p][0] = u.x; rb[p][1] = u.y; rb[p][2] = u.z; rb[p][3] = u.w;
                okb[p] = rowb[p] && kin;
            } else {
                load_w_mixed<4>(a, col_t + crow + RSTEP * p, k0 + ck, rb[p], okb[p]);
            }
        }
    };
    auto stage = [&](const float (&ra)[QA][4], const bool (&oka)[QA], const float (&rb)[QB][4],
                     const bool (&okb)[QB], int buf) {
#pragma unroll
        for (int p = 0; p < QA; ++p)
            *reinterpret_cast<float4*>(&As[buf][(crow + RSTEP * p) * LW + ck]) =
                oka[p] ? make_float4(ra[p][0], ra[p][1], ra[p][2], ra[p][3]) : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int p = 0; p < QB; ++p)
            *reinterpret_cast<float4*>(&Bs[buf][(crow + RSTEP * p) * LW + ck]) =
                okb[p] ? make_float4(rb[p][0], rb[p][1], rb[p][2], rb[p][3]) : make_float4(0.f, 0.f, 0.f, 0.f);
    };
    const int hk = HK * (lane >> 5);
    // A slice is consumed in groups of four k steps: the operand reads of
    // group q + 1 are issued before the MFMAs of group q, so only the first
    // group's LDS latency is exposed (all waves read right after the barrier).
    auto compute = [&](int buf) {
        float av[TM][HK], bv[TN][HK];
        auto read = [&](int q) {
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                const float4 u = reinterpret_cast<const float4*>(
                    &As[buf][(wm * WRM + i * 32 + (lane & 31)) * LW + hk])[q];
                av[i][4 * q] = u.x; av[i][4 * q + 1] = u.y; av[i][4 * q + 2] = u.z; av[i][4 * q + 3] = u.w;
            }
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const float4 u = reinterpret_cast<const float4*>(
                    &Bs[buf][(wn * WRN + j * 32 + (lane & 31)) * LW + hk])[q];
                bv[j][4 * q] = u.x; bv[j][4 * q + 1] = u.y; bv[j][4 * q + 2] = u.z; bv[j][4 * q + 3] = u.w;
            }
        };
        read(0);
#pragma unroll
        for (int q = 0; q < HK / 4; ++q) {
            if (q + 1 < HK / 4) read(q + 1);
            __builtin_amdgcn_sched_barrier(0);   // next group's reads ahead of this group's MFMAs
#pragma unroll
            for (int kk = 4 * q; kk < 4 * q + 4; ++kk)
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[i][kk], bv[j][kk], acc[i][j], 0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);   // and the LDS stores that follow stay after them
        }
    };

    // Slices come in pairs (compute from LDS buffer 0 then 1), so buffers
    // and register stages are fixed per half and nothing rotates across
    // the loop edge; an odd last slice is computed after the loop.  Slices
    // past this range are fetched (zero-filled or clamped) and never
    // computed, so every load is unconditional.
    const int n_slices = (k_hi - k_lo + BK - 1) / BK;
    fetch(ra0, oka0, rb0, okb0, k_lo);
    stage(ra0, oka0, rb0, okb0, 0);
    fetch(ra1, oka1, rb1, okb1, k_lo + BK);
    __syncthreads();
    int k0 = k_lo;
    for (int t = 0; t + 1 < n_slices; t += 2, k0 += 2 * BK) {
        fetch(ra0, oka0, rb0, okb0, k0 + 2 * BK);
        compute(0);
        stage(ra1, oka1, rb1, okb1, 1);
        __syncthreads();
        fetch(ra1, oka1, rb1, okb1, k0 + 3 * BK);
        compute(1);
        stage(ra0, oka0, rb0, okb0, 0);
        __syncthreads();
    }
    if (n_slices & 1) compute(0);
    if constexpr (SPLIT) {
        // staged columns past cc are zero, so four fused steps add exactly
        // the cc products
        if (blockIdx.z == 0) {
            float4 wc[TN];
#pragma unroll
            for (int j = 0; j < TN; ++j)
                wc[j] = *reinterpret_cast<const float4*>(&sWc[(wn * WRN + j * 32 + (lane & 31)) * 4]);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const float4 xr = *reinterpret_cast<const float4*>(
                        &sXc[(wm * WRM + i * 32 + 4 * (lane >> 5) + 8 * (r >> 2) + (r & 3)) * 4]);
#pragma unroll
                    for (int j = 0; j < TN; ++j) {
                        float t = acc[i][j][r];
                        t = fmaf(xr.x, wc[j].x, t);
                        t = fmaf(xr.y, wc[j].y, t);
                        t = fmaf(xr.z, wc[j].z, t);
                        t = fmaf(xr.w, wc[j].w, t);
                        acc[i][j][r] = t;
                    }
                }
        }
    }
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
            epilogue<EPI, false>(a, acc[i][j], row_t + wm * WRM + i * 32, col_t + wn * WRN + j * 32, lane);
}

// bf16 MFMA GEMM, same structure with k-slices of 32 and row-major LDS
// tiles (8 consecutive k per lane per MFMA operand).
template <int BM, int BN, int EPI, bool FAST_A, bool FAST_W>
__global__ __launch_bounds__(256) void gemm_bf16_kernel(GemmArgs a) {
    clear_pool_target(a);
    constexpr int BK = BKH;
    constexpr int TM = BM / 64, TN = BN / 64;
    constexpr int PA = BM / 64, PB = BN / 64;   // 8-element runs per thread per slice
    __shared__ __attribute__((aligned(16))) uint16_t As[2][BM * kRowH];
    __shared__ __attribute__((aligned(16))) uint16_t Bs[2][BN * kRowH];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int64_t row_t = (int64_t)blockIdx.x * BM;
    const int col_t = blockIdx.y * BN;
    const int lr = tid >> 2, lc = tid & 3, lk = lc * 8;   // 64 rows x 32 k per pass
    const int k_lo = blockIdx.z * a.kc;
    const int k_hi = min(a.K, k_lo + a.kc);

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    uint4 qa[PA], qb[PB];
    bool oka[PA], okb[PB];
#pragma unroll
    for (int p = 0; p < PA; ++p) qa[p] = load_a8_bf16<FAST_A>(a, row_t + lr + 64 * p, k_lo + lk, oka[p]);
#pragma unroll
    for (int p = 0; p < PB; ++p) qb[p] = load_w8_bf16<FAST_W>(a, col_t + lr + 64 * p, k_lo + lk, okb[p]);
#pragma unroll
    for (int p = 0; p < PA; ++p)
        *reinterpret_cast<uint4*>(&As[0][(lr + 64 * p) * kRowH + bf16_chunk(lr + 64 * p, lc)]) = select_u4(oka[p], qa[p]);
#pragma unroll
    for (int p = 0; p < PB; ++p)
        *reinterpret_cast<uint4*>(&Bs[0][(lr + 64 * p) * kRowH + bf16_chunk(lr + 64 * p, lc)]) = select_u4(okb[p], qb[p]);
    __syncthreads();

    int cur = 0;
    for (int k0 = k_lo; k0 < k_hi; k0 += BK) {
        // unconditional prefetch of the next slice (zero-filled past K)
#pragma unroll
        for (int p = 0; p < PA; ++p) qa[p] = load_a8_bf16<FAST_A>(a, row_t + lr + 64 * p, k0 + BK + lk, oka[p]);
#pragma unroll
        for (int p = 0; p < PB; ++p) qb[p] = load_w8_bf16<FAST_W>(a, col_t + lr + 64 * p, k0 + BK + lk, okb[p]);
        bf16x8 av[BK / 16][TM], bv[BK / 16][TN];
#pragma unroll
        for (int kk = 0; kk < BK / 16; ++kk) {
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                const int r = wm * (BM / 2) + i * 32 + (lane & 31);
                av[kk][i] = *reinterpret_cast<const bf16x8*>(&As[cur][r * kRowH + bf16_chunk(r, 2 * kk + (lane >> 5))]);
            }
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int r = wn * (BN / 2) + j * 32 + (lane & 31);
                bv[kk][j] = *reinterpret_cast<const bf16x8*>(&Bs[cur][r * kRowH + bf16_chunk(r, 2 * kk + (lane >> 5))]);
            }
        }
        __builtin_amdgcn_sched_barrier(0);   // keep the operand reads ahead of the MFMAs
#pragma unroll
        for (int kk = 0; kk < BK / 16; ++kk)
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[kk][i], bv[kk][j], acc[i][j], 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);   // next slice's LDS stores after all MFMAs
#pragma unroll
        for (int p = 0; p < PA; ++p)
            *reinterpret_cast<uint4*>(&As[cur ^ 1][(lr + 64 * p) * kRowH + bf16_chunk(lr + 64 * p, lc)]) =
                select_u4(oka[p], qa[p]);
#pragma unroll
        for (int p = 0; p < PB; ++p)
            *reinterpret_cast<uint4*>(&Bs[cur ^ 1][(lr + 64 * p) * kRowH + bf16_chunk(lr + 64 * p, lc)]) =
                select_u4(okb[p], qb[p]);
        __syncthreads();
        cur ^= 1;
    }
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
            epilogue<EPI, true>(a, acc[i][j], row_t + wm * (BM / 2) + i * 32, col_t + wn * (BN / 2) + j * 32, lane);
}

// Split-K finish: sum the partial products in split order (deterministic),
// then bias / ReLU / rounding and the store or pooled max.
template <int EPI>
__global__ __launch_bounds__(256) void splitk_finish_kernel(GemmArgs a, int splits) {
    const int64_t n = a.rows * a.N;
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < n; e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t row = e / a.N;
        const int col = (int)(e - row * a.N);
        float t = 0.0f;
        for (int z = 0; z < splits; ++z) t += a.part[(int64_t)z * n + e];
        const float v = a.round_bf16 ? activate<true>(a, t, a.bias ? a.bias[col] : 0.0f)
                                     : activate<false>(a, t, a.bias ? a.bias[col] : 0.0f);
        if constexpr (EPI == EPI_POOL)
            atomicMax(static_cast<unsigned*>(a.y) + (row / a.G) * a.ldy + col, __float_as_uint(v));
        else if constexpr (EPI == EPI_F32)
            static_cast<float*>(a.y)[row * a.ldy + col] = v;
        else
            static_cast<uint16_t*>(a.y)[row * a.ldy + col] = f32_to_bf16(v);
    }
}

// Skinny layers: at most 64 rows (the classifier head runs on one row per
// cloud).  A row-block GEMM would leave almost every CU idle and split K
// through partial sums; here a workgroup owns 16 output columns for all
// rows, its four waves split K, each accumulating 16 x 16 blocks with
// v_mfma_f32_16x16x4_f32 from operands loaded straight from L2 (lane l:
// row or column l % 16, k offset 4 (l / 16) inside a 16-wide chunk, one
// 16-byte load per operand and chunk, the MFMA steps consuming its four
// words), loads issued one group of chunks ahead.  The partial blocks are
// summed in wave order through LDS (deterministic), then bias and ReLU.
// The accumulator of a 16 x 16 MFMA holds, in lane l and register r, row
// 4 (l / 16) + r and column l % 16.
constexpr int kSkinnyRows = 64;
constexpr int kSkinnyWaves = 4;
typedef float f32x4 __attribute__((ext_vector_type(4)));

template <int TM>
__global__ __launch_bounds__(64 * kSkinnyWaves) void skinny_f32_kernel(const float* __restrict__ x, int64_t ldx, int rows, int K,
                                                         const float* __restrict__ W, const float* __restrict__ bias,
                                                         int N, int relu, float* __restrict__ y, int64_t ldy) {
    constexpr int G = 4;   // 16-wide k chunks per load group
    constexpr int NW = kSkinnyWaves;
    __shared__ float red[NW][TM * 4][64];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int i = lane & 15, q = lane >> 4;
    const int col0 = blockIdx.x * 16;
    const bool col_ok = col0 + i < N;
    const float* wr = W + (int64_t)(col_ok ? col0 + i : 0) * K;
    const float* xr[TM];
    bool rok[TM];
#pragma unroll
    for (int t = 0; t < TM; ++t) {
        const int r = 16 * t + i;
        rok[t] = r < rows;
        xr[t] = x + (int64_t)(rok[t] ? r : 0) * ldx;
    }
    const int nch = (K + 15) / 16;
    const int per = (nch + NW - 1) / NW;
    const int c_lo = min(nch, wave * per), c_hi = min(nch, c_lo + per);
    const int ngroups = (c_hi - c_lo + G - 1) / G;

    f32x4 acc[TM];
#pragma unroll
    for (int t = 0; t < TM; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    f32x4 la0[G][TM], lb0[G], la1[G][TM], lb1[G];
    const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
    // chunks past this wave's range or past K load column 0 and are zeroed
    auto load = [&](f32x4 (&la)[G][TM], f32x4 (&lb)[G], int c0) {
#pragma unroll
        for (int g = 0; g < G; ++g) {
            const int k = 16 * (c0 + g) + 4 * q;
            const bool in = c0 + g < c_hi && k < K;
            const int ko = in ? k : 0;
            const f32x4 u = *reinterpret_cast<const f32x4*>(wr + ko);
            lb[g] = (in && col_ok) ? u : zero;
#pragma unroll
            for (int t = 0; t < TM; ++t) {
                const f32x4 v = *reinterpret_cast<const f32x4*>(xr[t] + ko);
                la[g][t] = (in && rok[t]) ? v : zero;
            }
        }
    };
    auto compute = [&](const f32x4 (&la)[G][TM], const f32x4 (&lb)[G]) {
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
            for (int kk = 0; kk < 4; ++kk)
#pragma unroll
                for (int t = 0; t < TM; ++t)
                    acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(la[g][t][kk], lb[g][kk], acc[t], 0, 0, 0);
    };
    int c = c_lo;
    load(la0, lb0, c);
    load(la1, lb1, c + G);
    for (int t = 0; t + 1 < ngroups; t += 2, c += 2 * G) {
        compute(la0, lb0);
        load(la0, lb0, c + 2 * G);
        compute(la1, lb1);
        load(la1, lb1, c + 3 * G);
    }
    if (ngroups & 1) compute(la0, lb0);

#pragma unroll
    for (int t = 0; t < TM; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r) red[wave][4 * t + r][lane] = acc[t][r];
    __syncthreads();
    for (int o = tid; o < TM * 4 * 64; o += 64 * NW) {
        const int tr = o >> 6, l = o & 63;
        float sum = 0.0f;
#pragma unroll
        for (int w = 0; w < NW; ++w) sum += red[w][tr][l];
        const int row = 16 * (tr >> 2) + 4 * (l >> 4) + (tr & 3);
        const int cc = col0 + (l & 15);
        if (row < rows && cc < N) {
            float v = sum + (bias ? bias[cc] : 0.0f);
            if (relu) v = v > 0.0f ? v : 0.0f;
            y[(int64_t)row * ldy + cc] = v;
        }
    }
}

static int launch_skinny(const float* x, int64_t ldx, int rows, int K, const float* W, const float* bias, int N,
                         int relu, float* y, int64_t ldy, hipStream_t s) {
    const dim3 grid((unsigned)ceil_div(N, 16)), block(64 * kSkinnyWaves);
    const int tm = (int)ceil_div(rows, 16);
    if (tm == 1) skinny_f32_kernel<1><<<grid, block, 0, s>>>(x, ldx, rows, K, W, bias, N, relu, y, ldy);
    else if (tm == 2) skinny_f32_kernel<2><<<grid, block, 0, s>>>(x, ldx, rows, K, W, bias, N, relu, y, ldy);
    else if (tm == 3) skinny_f32_kernel<3><<<grid, block, 0, s>>>(x, ldx, rows, K, W, bias, N, relu, y, ldy);
    else skinny_f32_kernel<4><<<grid, block, 0, s>>>(x, ldx, rows, K, W, bias, N, relu, y, ldy);
    return after_launch("mesorasi_pointwise_mlp");
}

// The skinny path takes fp32 MLPs on at most 64 rows with one 16-byte
// aligned input source, layer widths that are multiples of 4, 16-byte
// aligned weights, fp32 output and no pooling.
static bool skinny_ok(const float* x0, int64_t ld0, const float* x1, int c1, int64_t rows, int n_layers,
                      const int32_t* dims, const void* const* W, int dtype, int out_dtype, int64_t pool_group) {
    if (dtype != MESORASI_F32 || out_dtype != MESORASI_F32 || pool_group > 0) return false;
    if (rows < 1 || rows > kSkinnyRows || c1 != 0 || x1 != nullptr) return false;
    if (ld0 % 4 != 0 || !aligned(x0, 16)) return false;
    for (int l = 0; l < n_layers; ++l)
        if (dims[l] % 4 != 0 || !aligned(W[l], 16)) return false;
    return true;
}

struct LayerPlan {
    int bm, bn, bk, splits, kc;
};

// fp32 k-slice depth for a tile: about 2K MFMA cycles per slice and wave
// (TM x TN blocks x BK/2 MFMAs of 64 cycles), enough to cover the latency of
// the next slice's global loads.
static int f32_slice(int bm, int bn) { return (bm / 64) * (bn / 64) >= 2 ? 32 : 64; }

// Tile shape and K split of one layer: a pure function of the shape, shared
// by the workspace query and the launch.  Picks the tile with the smallest
// estimated makespan (tile rounds x tile area) and, when even 64 x 64 tiles
// leave most CUs idle, splits K.
static LayerPlan plan_layer(int64_t rows, int N, int K, bool bf16) {
    static const int cand[4][2] = {{128, 128}, {128, 64}, {64, 128}, {64, 64}};
    LayerPlan best{64, 64, 0, 1, K};
    double best_cost = 1e300;
    for (const auto& c : cand) {
        const int64_t tiles = ceil_div(rows, c[0]) * ceil_div(N, c[1]);
        const double cost = (double)ceil_div(tiles, kTargetTiles) * c[0] * c[1];
        if (cost < best_cost * (1.0 - 1e-9)) {
            best_cost = cost;
            best = {c[0], c[1], 0, 1, K};
        }
    }
    best.bk = bf16 ? BKH : f32_slice(best.bm, best.bn);
    const int bk = best.bk;
    const int64_t tiles = ceil_div(rows, best.bm) * ceil_div(N, best.bn);
    if (tiles < kTargetTiles / 2) {
        int splits = 1;
        while (tiles * splits * 2 <= kTargetTiles && K / (splits * 2) >= 4 * bk) splits *= 2;
        if (splits > 1) {
            const int kc = (int)ceil_div(ceil_div(K, splits), bk) * bk;
            best.splits = (int)ceil_div(K, kc);
            best.kc = kc;
        }
    }
    return best;
}

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Workspace: two ping-pong buffers for the intermediate activations, then
// the split-K partial sums of the largest split layer.
struct MlpWs {
    size_t act, part;
};
static MlpWs mlp_ws_layout(int64_t rows, int n_layers, const int32_t* dims, int dtype) {
    MlpWs w{0, 0};
    if (rows <= 0) return w;
    int64_t width = 0;
    for (int l = 1; l < n_layers; ++l) width = std::max<int64_t>(width, dims[l]);
    const size_t elem = dtype == MESORASI_BF16 ? 2 : 4;
    const size_t one = align256((size_t)rows * (size_t)width * elem);
    w.act = n_layers <= 1 ? 0 : (n_layers == 2 ? one : 2 * one);
    for (int l = 0; l < n_layers; ++l) {
        const LayerPlan pl = plan_layer(rows, dims[l + 1], dims[l], dtype == MESORASI_BF16);
        if (pl.splits > 1) w.part = std::max(w.part, align256((size_t)pl.splits * rows * dims[l + 1] * 4));
    }
    return w;
}
// The fused narrow kernel or the layer-by-layer GEMM (measured on MI355X):
// the fused kernel wins on neighbour rows gathered in its loader (the
// conventional and limited modules) and on up to 32768 plain rows (32768 x
// 3 -> 64 -> 64 -> 128: 21.0 against 24.2 us); above, the GEMM's larger
// tiles win (65536 x 131 -> 128 -> 128 -> 128: 102 against 127 us; 65536 x
// 128 -> 128 -> 13: 45 against 71 us; 65536 x 6 -> 32 -> 32 -> 64: 22.6
// against 27.2 us).
constexpr int64_t kFusedMaxPlainRows = 32768;
static bool use_fused(int64_t rows, int n_layers, const int32_t* dims, int dtype, bool neighbor_rows) {
    return fused_mlp_supported(n_layers, dims, dtype) && (neighbor_rows || rows <= kFusedMaxPlainRows);
}

// The register-resident MLP (mlp_rr.hip, mlp_rr_bf16.hip) for plain rows
// above that count when every layer is at most 128 wide; in bf16 only for
// first layers of at most 32 inputs, where the GEMM's per-layer launches
// and HBM round trips dominate (65536 x 3 -> 32 -> 32 -> 64: 16.6 against
// 20.8 us); on 128-wide rows the bf16 GEMM is faster (65536 x 128 -> 128
// -> 128: 28.5 against 34.7 us), its MFMA work being a sixteenth of fp32's.
#ifndef MESO_RR_MIN_ROWS
#define MESO_RR_MIN_ROWS (kFusedMaxPlainRows + 1)
#endif
static bool use_rr(int64_t rows, int n_layers, const int32_t* dims, int dtype, int out_dtype, int64_t pool_group,
                   bool neighbor_rows) {
    if (pool_group != 0 || neighbor_rows || rows < MESO_RR_MIN_ROWS) return false;
    if (dtype == MESORASI_F32) return out_dtype == MESORASI_F32 && rr_mlp_supported(n_layers, dims, rows);
    return dtype == MESORASI_BF16 && dims[0] <= 32 && rb_mlp_supported(n_layers, dims);
}

static size_t mlp_ws_bytes(int64_t rows, int n_layers, const int32_t* dims, int dtype, bool neighbor_rows) {
    if (use_fused(rows, n_layers, dims, dtype, neighbor_rows)) return 0;
    const MlpWs w = mlp_ws_layout(rows, n_layers, dims, dtype);
    return w.act + w.part;
}

// fp32 tiles run with NW waves in an (NW / 2) x 2 grid; bf16 tiles with four.
template <int BM, int BN, int EPI, int NW = 4>
static void launch_tile(const GemmArgs& a, bool bf16, bool fast_a, bool fast_w, dim3 grid, hipStream_t s) {
    const dim3 block(256), fblock(64 * NW);
    constexpr int BK = (BM / 64) * (BN / 64) >= 2 ? 32 : 64;   // f32_slice(BM, BN)
    if (a.cc > 0) {
        gemm_f32_kernel<BM, BN, BK, EPI, true, false, true, false, NW><<<grid, fblock, 0, s>>>(a);
        return;
    }
    if (a.lq) {
        gemm_f32_kernel<BM, BN, BK, EPI, true, true, false, true, NW><<<grid, fblock, 0, s>>>(a);
        return;
    }
    if (bf16) {
        if (fast_a && fast_w) gemm_bf16_kernel<BM, BN, EPI, true, true><<<grid, block, 0, s>>>(a);
        else if (fast_w) gemm_bf16_kernel<BM, BN, EPI, false, true><<<grid, block, 0, s>>>(a);
        else gemm_bf16_kernel<BM, BN, EPI, false, false><<<grid, block, 0, s>>>(a);
    } else {
        if (fast_a && fast_w) gemm_f32_kernel<BM, BN, BK, EPI, true, true, false, false, NW><<<grid, fblock, 0, s>>>(a);
        else if (fast_w) gemm_f32_kernel<BM, BN, BK, EPI, false, true, false, false, NW><<<grid, fblock, 0, s>>>(a);
        else gemm_f32_kernel<BM, BN, BK, EPI, false, false, false, false, NW><<<grid, fblock, 0, s>>>(a);
    }
}

// 128 x 128 and 128 x 64 fp32 tiles run with eight waves (two per SIMD,
// 32 x 64 or 32 x 32 each), so one wave's LDS and barrier waits overlap the
// other's MFMAs; with a full wave of 256 x 128 tiles (plain fast sources, no
// split K) the tile doubles to 64 x 64 per wave, halving the staged B
// traffic per row.
template <int EPI>
static void launch_epi(const GemmArgs& a, const LayerPlan& pl, bool bf16, bool fast_a, bool fast_w, hipStream_t s) {
    if (pl.bm == 128 && pl.bn == 128 && pl.splits == 1 && !bf16 && fast_a && fast_w && a.cc == 0 && !a.lq &&
        ceil_div(a.rows, 256) * ceil_div(a.N, 128) >= kTargetTiles) {
        const dim3 g8((unsigned)ceil_div(a.rows, 256), (unsigned)ceil_div(a.N, 128), 1);
        gemm_f32_kernel<256, 128, 32, EPI, true, true, false, false, 8><<<g8, dim3(512), 0, s>>>(a);
        return;
    }
    const dim3 grid((unsigned)ceil_div(a.rows, pl.bm), (unsigned)ceil_div(a.N, pl.bn), (unsigned)pl.splits);
    if (pl.bm == 128 && pl.bn == 128) {
        if (bf16) launch_tile<128, 128, EPI>(a, bf16, fast_a, fast_w, grid, s);
        else launch_tile<128, 128, EPI, 8>(a, bf16, fast_a, fast_w, grid, s);
    }
    else if (pl.bm == 128) {
        if (bf16) launch_tile<128, 64, EPI>(a, bf16, fast_a, fast_w, grid, s);
        else launch_tile<128, 64, EPI, 8>(a, bf16, fast_a, fast_w, grid, s);
    }
    else if (pl.bn == 128) launch_tile<64, 128, EPI>(a, bf16, fast_a, fast_w, grid, s);
    else launch_tile<64, 64, EPI>(a, bf16, fast_a, fast_w, grid, s);
}

// Launch one layer.  epi: EPI_F32 / EPI_BF16 / EPI_POOL.
static bool split_ok(const GemmArgs& a, bool bf16) {
    return !bf16 && !a.a_bf16 && a.x1 && a.c1 > 0 && a.c0 <= 4 && a.c1 % 4 == 0 && a.ld1 % 4 == 0 &&
           aligned(a.x1, 16) && aligned(a.W, 4);
}

static int launch_layer(GemmArgs a, bool bf16, int epi, float* part, hipStream_t s) {
    a.ldw = a.K;
    const bool split = split_ok(a, bf16);
    MESO_REQUIRE(split || !a.gnit || a.lq, MESORASI_EUNSUPPORTED, "gathered layer without the split form");
    if (split) {
        // split form: the k loop over x1 alone, x0 added in the epilogue
        a.xc = static_cast<const float*>(a.x0);
        a.ldc = a.ld0;
        a.cc = a.c0;
        a.x0 = a.x1;
        a.ld0 = a.ld1;
        a.c0 = a.c1;
        a.x1 = nullptr;
        a.ld1 = 0;
        a.c1 = 0;
        a.W = static_cast<const float*>(a.W) + a.cc;
        a.K = a.c0;
    }
    const LayerPlan pl = plan_layer(a.rows, a.N, a.K, bf16);
    a.kc = pl.kc;
    // vector loads: 16-byte aligned rows and whole 16-byte chunks (4 fp32
    // per chunk in the fp32 kernel, 8 bf16 in the bf16 kernel)
    const int kq = bf16 ? 8 : 4;
    const bool fast_w = (a.K % kq == 0) && aligned(a.W, 16);
    bool fast_a;
    if (a.a_bf16) fast_a = a.c1 == 0 && a.c0 == a.K && a.K % 8 == 0 && a.ld0 % 8 == 0 && aligned(a.x0, 16);
    else fast_a = a.c1 == 0 && a.c0 == a.K && a.K % kq == 0 && a.ld0 % 4 == 0 && aligned(a.x0, 16);
    MESO_REQUIRE(!a.lq || (!bf16 && fast_a && fast_w), MESORASI_EUNSUPPORTED, "gathered layer without fast operands");
    if (pl.splits > 1) {
        a.part = part;
        launch_epi<EPI_PARTIAL>(a, pl, bf16, fast_a, fast_w, s);
        int rc = after_launch("mesorasi_pointwise_mlp");
        if (rc != MESORASI_OK) return rc;
        const int64_t n = a.rows * a.N;
        const dim3 grid((unsigned)std::min<int64_t>(ceil_div(n, 256), 4096)), block(256);
        if (epi == EPI_POOL) splitk_finish_kernel<EPI_POOL><<<grid, block, 0, s>>>(a, pl.splits);
        else if (epi == EPI_F32) splitk_finish_kernel<EPI_F32><<<grid, block, 0, s>>>(a, pl.splits);
        else splitk_finish_kernel<EPI_BF16><<<grid, block, 0, s>>>(a, pl.splits);
        return after_launch("mesorasi_pointwise_mlp");
    }
    if (epi == EPI_POOL) launch_epi<EPI_POOL>(a, pl, bf16, fast_a, fast_w, s);
    else if (epi == EPI_F32) launch_epi<EPI_F32>(a, pl, bf16, fast_a, fast_w, s);
    else launch_epi<EPI_BF16>(a, pl, bf16, fast_a, fast_w, s);
    return after_launch("mesorasi_pointwise_mlp");
}

static int check_mlp_spec(const char* who, int64_t rows, int n_layers, const int32_t* dims, int dtype) {
    MESO_REQUIRE(rows >= 0, MESORASI_EINVAL, "%s: rows < 0", who);
    MESO_REQUIRE(dims != nullptr, MESORASI_EINVAL, "%s: NULL dims", who);
    MESO_REQUIRE(n_layers >= 1 && n_layers <= MESORASI_MAX_LAYERS, MESORASI_EUNSUPPORTED, "%s: n_layers = %d", who,
                 n_layers);
    for (int l = 0; l <= n_layers; ++l) {
        MESO_REQUIRE(dims[l] >= 1, MESORASI_EINVAL, "%s: dims[%d] = %d < 1", who, l, dims[l]);
        MESO_REQUIRE(dims[l] <= MESORASI_MAX_WIDTH, MESORASI_EUNSUPPORTED, "%s: dims[%d] = %d > %d", who, l, dims[l],
                     MESORASI_MAX_WIDTH);
    }
    MESO_REQUIRE(dtype == MESORASI_F32 || dtype == MESORASI_BF16, MESORASI_EUNSUPPORTED, "%s: dtype %d", who, dtype);
    return MESORASI_OK;
}

// The MLP proper, after validation.
static int run_mlp(const float* x0, int c0, int64_t ld0, const float* x1, int c1, int64_t ld1, int64_t rows,
                   int n_layers, const int32_t* dims, const void* const* W, const float* const* bias,
                   uint32_t relu_mask, int dtype, int out_dtype, void* y, int64_t ld_y, int64_t pool_group, void* ws,
                   hipStream_t s, bool neighbor_rows, const MlpGather* g = nullptr) {
    if (!g && use_rr(rows, n_layers, dims, dtype, out_dtype, pool_group, neighbor_rows)) {
        if (dtype == MESORASI_BF16)
            return run_rb_mlp(x0, c0, ld0, x1, c1, ld1, rows, n_layers, dims, W, bias, relu_mask, out_dtype, y, ld_y,
                              s);
        return run_rr_mlp(x0, c0, ld0, x1, c1, ld1, rows, n_layers, dims, W, bias, relu_mask, static_cast<float*>(y),
                          ld_y, s);
    }
    if (use_fused(rows, n_layers, dims, dtype, neighbor_rows))
        return run_fused_mlp(x0, c0, ld0, x1, c1, ld1, rows, n_layers, dims, W, bias, relu_mask, out_dtype, y, ld_y,
                             pool_group, s, g);
    const bool bf16 = dtype == MESORASI_BF16;
    const size_t elem = bf16 ? 2 : 4;
    int64_t w = 0;
    for (int l = 1; l < n_layers; ++l) w = std::max<int64_t>(w, dims[l]);
    const size_t one = align256((size_t)rows * (size_t)w * elem);
    const MlpWs lay = mlp_ws_layout(rows, n_layers, dims, dtype);
    char* buf[2] = {static_cast<char*>(ws), static_cast<char*>(ws) + one};
    if (!g && skinny_ok(x0, ld0, x1, c1, rows, n_layers, dims, W, dtype, out_dtype, pool_group)) {
        // uses only the activation part of the workspace
        for (int l = 0; l < n_layers; ++l) {
            const float* xin = l == 0 ? x0 : reinterpret_cast<const float*>(buf[(l - 1) & 1]);
            const int64_t ldx = l == 0 ? ld0 : dims[l];
            const bool last = l + 1 == n_layers;
            float* yout = last ? static_cast<float*>(y) : reinterpret_cast<float*>(buf[l & 1]);
            const int64_t ldo = last ? ld_y : dims[l + 1];
            const int rc = launch_skinny(xin, ldx, (int)rows, dims[l], static_cast<const float*>(W[l]),
                                         bias ? bias[l] : nullptr, dims[l + 1], (relu_mask >> l) & 1u, yout, ldo, s);
            if (rc != MESORASI_OK) return rc;
        }
        return MESORASI_OK;
    }
    float* part = reinterpret_cast<float*>(static_cast<char*>(ws) + lay.act);
    // a pooled multi-layer MLP clears its output from the first layer's
    // kernel; a single pooled layer needs the fill launch first
    if (pool_group > 0 && n_layers == 1) {
        const int rc = zero_rows_f32(static_cast<float*>(y), rows / pool_group, dims[n_layers], ld_y, s);
        if (rc != MESORASI_OK) return rc;
    }
    for (int l = 0; l < n_layers; ++l) {
        GemmArgs a{};
        if (l == 0) {
            a.x0 = x0; a.ld0 = ld0; a.x1 = x1; a.ld1 = ld1; a.c0 = c0; a.c1 = c1; a.a_bf16 = 0;
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
            if (pool_group > 0 && n_layers > 1) {
                a.zy = static_cast<float*>(y);
                a.zrows = rows / pool_group;
                a.zcols = dims[n_layers];
                a.zld = ld_y;
            }
        } else {
            a.x0 = buf[(l - 1) & 1]; a.ld0 = dims[l]; a.x1 = nullptr; a.ld1 = 0; a.c0 = dims[l]; a.c1 = 0;
            a.a_bf16 = bf16 ? 1 : 0;
        }
        a.rows = rows;
        a.K = dims[l];
        a.N = dims[l + 1];
        a.W = W[l];
        a.bias = bias ? bias[l] : nullptr;
        a.relu = (relu_mask >> l) & 1u;
        a.round_bf16 = bf16 ? 1 : 0;
        int epi;
        if (l + 1 < n_layers) {
            a.y = buf[l & 1];
            a.ldy = dims[l + 1];
            epi = bf16 ? EPI_BF16 : EPI_F32;
        } else {
            a.y = y;
            a.ldy = ld_y;
            a.G = pool_group;
            epi = pool_group > 0 ? EPI_POOL : (out_dtype == MESORASI_BF16 ? EPI_BF16 : EPI_F32);
        }
        const int rc = launch_layer(a, bf16, epi, part, s);
        if (rc != MESORASI_OK) return rc;
    }
    return MESORASI_OK;
}

// ---------------------------------------------------------------------------
// conventional module: neighbor feature matrix, then the MLP with pooling
// ---------------------------------------------------------------------------

__global__ void group_pointnet_kernel(const float* __restrict__ xyz, const float* __restrict__ feat, int cf,
                                      int64_t ldf, const float* __restrict__ cxyz, const int32_t* __restrict__ nit,
                                      int N, int M, int K, int64_t total_rows, float* __restrict__ nfm) {
    const int cin = 3 + cf;
    const int64_t n = total_rows * cin;
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < n; e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t row = e / cin;
        const int c = (int)(e - row * cin);
        const int64_t cm = row / K;   // global centroid (b*M + m)
        const int64_t b = cm / M;
        const int64_t j = b * N + nit[row];
        nfm[e] = c < 3 ? xyz[j * 3 + c] - cxyz[cm * 3 + c] : feat[j * ldf + (c - 3)];
    }
}

__global__ void group_edge_kernel(const float* __restrict__ f, int C, int64_t ldf, const int32_t* __restrict__ nit,
                                  int N, int K, int64_t total_rows, float* __restrict__ nfm) {
    const int cin = 2 * C;
    const int64_t n = total_rows * cin;
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < n; e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t row = e / cin;
        const int c = (int)(e - row * cin);
        const int64_t i = row / K;    // global point (b*N + i)
        const int64_t b = i / N;
        const float fi = f[i * ldf + (c < C ? c : c - C)];
        if (c < C) {
            nfm[e] = fi;
        } else {
            const int64_t j = b * N + nit[row];
            nfm[e] = f[j * ldf + (c - C)] - fi;
        }
    }
}

// First layer of a limited-delayed module (Sec. 7.3): every (centroid,
// neighbor) row h1 = ReLU(p1[neighbor] - q[centroid] + b1), four channels
// per thread when the rows allow 16-byte access.
template <bool VEC>
__global__ void ltd_group_kernel(const float* __restrict__ p1, int64_t ldp, const float* __restrict__ q, int64_t ldq,
                                 const float* __restrict__ b1, const int32_t* __restrict__ nit, int N, int M, int K,
                                 int C, int64_t total_rows, float* __restrict__ h1) {
    const int L = VEC ? 4 : 1;
    const int CL = C / L;
    const int64_t n = total_rows * CL;
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < n; e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t row = e / CL;
        const int c = (int)(e - row * CL) * L;
        const int64_t cm = row / K;            // global centroid (b * M + m)
        const int64_t b = cm / M;
        const int64_t j = b * N + nit[row];
        if constexpr (VEC) {
            const float4 pv = *reinterpret_cast<const float4*>(p1 + j * ldp + c);
            const float4 qv = *reinterpret_cast<const float4*>(q + cm * ldq + c);
            const float4 bv = b1 ? *reinterpret_cast<const float4*>(b1 + c) : make_float4(0.f, 0.f, 0.f, 0.f);
            float4 v;
            v.x = (pv.x - qv.x) + bv.x;
            v.y = (pv.y - qv.y) + bv.y;
            v.z = (pv.z - qv.z) + bv.z;
            v.w = (pv.w - qv.w) + bv.w;
            v.x = v.x > 0.0f ? v.x : 0.0f;
            v.y = v.y > 0.0f ? v.y : 0.0f;
            v.z = v.z > 0.0f ? v.z : 0.0f;
            v.w = v.w > 0.0f ? v.w : 0.0f;
            *reinterpret_cast<float4*>(h1 + row * C + c) = v;
        } else {
            const float v = (p1[j * ldp + c] - q[cm * ldq + c]) + (b1 ? b1[c] : 0.0f);
            h1[row * C + c] = v > 0.0f ? v : 0.0f;
        }
    }
}

}  // namespace meso

using namespace meso;

extern "C" size_t mesorasi_pointwise_mlp_workspace(int64_t rows, int32_t n_layers, const int32_t* dims, int32_t dtype,
                                                   int64_t pool_group) {
    (void)pool_group;
    if (check_mlp_spec("mesorasi_pointwise_mlp_workspace", rows, n_layers, dims, dtype) != MESORASI_OK) return 0;
    return mlp_ws_bytes(rows, n_layers, dims, dtype, false);
}

// Argument checks shared by both MLP entry points (host only, no HIP call).
static int check_mlp_args(const char* who, const float* x0, int32_t c0, int64_t ld0, const float* x1, int32_t c1,
                          int64_t ld1, int64_t rows, int32_t n_layers, const int32_t* dims, const void* const* W,
                          uint32_t relu_mask, int32_t dtype, int32_t out_dtype, void* y, int64_t ld_y,
                          int64_t pool_group) {
    int rc = check_mlp_spec(who, rows, n_layers, dims, dtype);
    if (rc != MESORASI_OK) return rc;
    MESO_REQUIRE(c0 >= 1 && c1 >= 0, MESORASI_EINVAL, "%s: c0 = %d, c1 = %d", who, c0, c1);
    MESO_REQUIRE(ld0 >= c0 && (c1 == 0 || ld1 >= c1), MESORASI_EINVAL, "%s: leading dimension < width", who);
    MESO_REQUIRE(dims[0] == c0 + c1, MESORASI_EINVAL, "%s: dims[0] = %d != c0 + c1 = %d", who, dims[0], c0 + c1);
    MESO_REQUIRE(ld_y >= dims[n_layers], MESORASI_EINVAL, "%s: ld_y < dims[n_layers]", who);
    MESO_REQUIRE(out_dtype == MESORASI_F32 || out_dtype == MESORASI_BF16, MESORASI_EUNSUPPORTED, "%s: out_dtype %d",
                 who, out_dtype);
    MESO_REQUIRE(pool_group >= 0, MESORASI_EINVAL, "%s: pool_group < 0", who);
    MESO_REQUIRE(pool_group <= 0x7fffffff, MESORASI_EUNSUPPORTED, "%s: pool_group > 2^31 - 1", who);
    if (pool_group > 0) {
        MESO_REQUIRE(rows % pool_group == 0, MESORASI_EINVAL, "%s: rows %% pool_group != 0", who);
        MESO_REQUIRE((relu_mask >> (n_layers - 1)) & 1u, MESORASI_EUNSUPPORTED, "%s: pooling needs a final ReLU", who);
        MESO_REQUIRE(out_dtype == MESORASI_F32, MESORASI_EUNSUPPORTED, "%s: pooling needs out_dtype F32", who);
    }
    if (rows == 0) return MESORASI_OK;
    MESO_REQUIRE(x0 && y && W, MESORASI_EINVAL, "%s: NULL x0, y or W", who);
    MESO_REQUIRE(c1 == 0 || x1, MESORASI_EINVAL, "%s: NULL x1 with c1 > 0", who);
    for (int l = 0; l < n_layers; ++l) MESO_REQUIRE(W[l] != nullptr, MESORASI_EINVAL, "%s: W[%d] is NULL", who, l);
    MESO_REQUIRE(rows / 64 < 0x7fffffff, MESORASI_EUNSUPPORTED, "%s: too many rows", who);
    return MESORASI_OK;
}

extern "C" int mesorasi_pointwise_mlp(const float* x0, int32_t c0, int64_t ld0, const float* x1, int32_t c1,
                                      int64_t ld1, int64_t rows, int32_t n_layers, const int32_t* dims,
                                      const void* const* W, const float* const* bias, uint32_t relu_mask,
                                      int32_t dtype, int32_t out_dtype, void* y, int64_t ld_y, int64_t pool_group,
                                      void* ws, size_t ws_bytes, void* stream) {
    const char* who = "mesorasi_pointwise_mlp";
    const int rc = check_mlp_args(who, x0, c0, ld0, x1, c1, ld1, rows, n_layers, dims, W, relu_mask, dtype,
                                  out_dtype, y, ld_y, pool_group);
    if (rc != MESORASI_OK || rows == 0) return rc;
    const size_t need = mlp_ws_bytes(rows, n_layers, dims, dtype, false);
    MESO_REQUIRE(ws_bytes >= need && (need == 0 || ws), MESORASI_EWORKSPACE, "%s: workspace %zu < %zu bytes", who,
                 ws_bytes, need);
    return run_mlp(x0, c0, ld0, x1, c1, ld1, rows, n_layers, dims, W, bias, relu_mask, dtype, out_dtype, y, ld_y,
                   pool_group, ws, as_stream(stream), false);
}

// ---------------------------------------------------------------------------
// allocation-free variant: the workspace is a file-scope device array
// ---------------------------------------------------------------------------

// Every GPU the library runs on holds its own copy until the process ends.
// In host code `scratch` names a host-side stand-in: kernels and copies get
// the device address from hipGetSymbolAddress, kept per device.
static __device__ __align__(256) unsigned char scratch[MESORASI_NOALLOC_WS_BYTES];

constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static void* g_scratch_dev[kMaxDevices];

// Device address of the current device's scratch array, looked up once per
// device (with that device current) on its first use.
static int scratch_on_current_device(const char* who, void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return set_error(MESORASI_EHIP, "%s: hipGetDevice: %s", who, hipGetErrorString(e));
    MESO_REQUIRE(dev >= 0 && dev < kMaxDevices, MESORASI_EUNSUPPORTED, "%s: device %d", who, dev);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_dev[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return set_error(MESORASI_EHIP, "%s: hipGetSymbolAddress(scratch): %s", who, hipGetErrorString(e));
        g_scratch_dev[dev] = p;
    }
    *out = g_scratch_dev[dev];
    return MESORASI_OK;
}

extern "C" int mesorasi_pointwise_mlp_noalloc(const float* x0, int32_t c0, int64_t ld0, const float* x1, int32_t c1,
                                              int64_t ld1, int64_t rows, int32_t n_layers, const int32_t* dims,
                                              const void* const* W, const float* const* bias, uint32_t relu_mask,
                                              int32_t dtype, int32_t out_dtype, void* y, int64_t ld_y,
                                              int64_t pool_group, void* stream) {
    const char* who = "mesorasi_pointwise_mlp_noalloc";
    int rc = check_mlp_args(who, x0, c0, ld0, x1, c1, ld1, rows, n_layers, dims, W, relu_mask, dtype, out_dtype, y,
                            ld_y, pool_group);
    if (rc != MESORASI_OK || rows == 0) return rc;
    const size_t need = mlp_ws_bytes(rows, n_layers, dims, dtype, false);
    MESO_REQUIRE(need <= (size_t)MESORASI_NOALLOC_WS_BYTES, MESORASI_EUNSUPPORTED,
                 "%s: needs %zu bytes of scratch, above the fixed %zu", who, need,
                 (size_t)MESORASI_NOALLOC_WS_BYTES);
    void* ws = nullptr;
    if (need > 0) {
        rc = scratch_on_current_device(who, &ws);
        if (rc != MESORASI_OK) return rc;
    }
    // the activations and split-K partials are written before they are
    // read, so nothing in the array needs clearing between calls
    return run_mlp(x0, c0, ld0, x1, c1, ld1, rows, n_layers, dims, W, bias, relu_mask, dtype, out_dtype, y, ld_y,
                   pool_group, ws, as_stream(stream), false);
}

extern "C" int mesorasi_aggregate_mlp(const float* cxyz, const float* pft, int64_t ld_pft, const int32_t* nit,
                                     const int32_t* cidx, int64_t B, int64_t N, int64_t M, int32_t K, int32_t C,
                                     int32_t n_layers, const int32_t* dims, const void* const* W,
                                     const float* const* bias, uint32_t relu_mask, float* y, int64_t ld_y,
                                     float* agg_out, int64_t ld_agg, void* stream) {
    const char* who = "mesorasi_aggregate_mlp";
    MESO_REQUIRE(B >= 0 && N >= 0 && M >= 0, MESORASI_EINVAL, "%s: negative size", who);
    MESO_REQUIRE(K >= 1, MESORASI_EINVAL, "%s: K = %d < 1", who, K);
    MESO_REQUIRE(C >= 1 && ld_pft >= C, MESORASI_EINVAL, "%s: C = %d, ld_pft = %lld", who, C, (long long)ld_pft);
    int rc = check_mlp_spec(who, B * M, n_layers, dims, MESORASI_F32);
    if (rc != MESORASI_OK) return rc;
    MESO_REQUIRE(dims[0] == 3 + C, MESORASI_EINVAL, "%s: dims[0] = %d != 3 + C = %d", who, dims[0], 3 + C);
    MESO_REQUIRE(ld_y >= dims[n_layers], MESORASI_EINVAL, "%s: ld_y < dims[n_layers]", who);
    MESO_REQUIRE(!agg_out || ld_agg >= C, MESORASI_EINVAL, "%s: ld_agg < C", who);
    MESO_REQUIRE(fused_mlp_supported(n_layers, dims, MESORASI_F32), MESORASI_EUNSUPPORTED,
                 "%s: the MLP is not a narrow fused one (at least 2 layers, inputs <= 160, outputs <= 128)", who);
    MESO_REQUIRE(C % 4 == 0 && ld_pft % 4 == 0 && (!agg_out || ld_agg % 4 == 0), MESORASI_EUNSUPPORTED,
                 "%s: C and the leading dimensions must be multiples of 4", who);
    if (B == 0 || M == 0) return MESORASI_OK;
    MESO_REQUIRE(N >= 1, MESORASI_EINVAL, "%s: N = 0 with M > 0", who);
    MESO_REQUIRE(cxyz && pft && nit && cidx && y && W, MESORASI_EINVAL, "%s: NULL pointer", who);
    for (int l = 0; l < n_layers; ++l) MESO_REQUIRE(W[l] != nullptr, MESORASI_EINVAL, "%s: W[%d] is NULL", who, l);
    MESO_REQUIRE(aligned(pft, 16) && (!agg_out || aligned(agg_out, 16)), MESORASI_EUNSUPPORTED,
                 "%s: pft and agg_out must be 16-byte aligned", who);
    MESO_REQUIRE((B * M) / 64 < 0x7fffffff, MESORASI_EUNSUPPORTED, "%s: too many rows", who);
    MlpAggregate ag{pft, ld_pft, N, M, nit, cidx, K, C, agg_out, ld_agg};
    return run_fused_aggregate_mlp(cxyz, ag, B * M, n_layers, dims, W, bias, relu_mask, y, ld_y, as_stream(stream));
}

extern "C" int mesorasi_interpolate3_mlp(const int32_t* nit, const float* dist, const float* f_src, int64_t ld_src,
                                         int64_t B, int64_t Nd, int64_t Ns, const float* add, int64_t ld_add,
                                         int32_t relu, int32_t n_layers, const int32_t* dims, const void* const* W,
                                         const float* const* bias, uint32_t relu_mask, float* y, int64_t ld_y,
                                         void* stream) {
    const char* who = "mesorasi_interpolate3_mlp";
    MESO_REQUIRE(B >= 0 && Nd >= 0 && Ns >= 0, MESORASI_EINVAL, "%s: negative size", who);
    int rc = check_mlp_spec(who, B * Nd, n_layers, dims, MESORASI_F32);
    if (rc != MESORASI_OK) return rc;
    const int C = dims[0];
    MESO_REQUIRE(ld_src >= C && ld_add >= C && ld_y >= dims[n_layers], MESORASI_EINVAL, "%s: leading dimension", who);
    MESO_REQUIRE(rr_mlp_supported(n_layers, dims, B * Nd), MESORASI_EUNSUPPORTED,
                 "%s: every layer must be at most 128 wide (the register-resident MLP), and layers whose "
                 "weights do not fit the LDS together need at most 32 rows per wave of the device", who);
    MESO_REQUIRE(C % 4 == 0 && ld_src % 4 == 0 && ld_add % 4 == 0, MESORASI_EUNSUPPORTED,
                 "%s: dims[0] and the leading dimensions of f_src and add must be multiples of 4", who);
    if (B == 0 || Nd == 0) return MESORASI_OK;
    MESO_REQUIRE(Ns >= 1, MESORASI_EINVAL, "%s: Ns = 0", who);
    MESO_REQUIRE(nit && dist && f_src && add && y && W, MESORASI_EINVAL, "%s: NULL pointer", who);
    for (int l = 0; l < n_layers; ++l) MESO_REQUIRE(W[l] != nullptr, MESORASI_EINVAL, "%s: W[%d] is NULL", who, l);
    MESO_REQUIRE(aligned(f_src, 16) && aligned(add, 16), MESORASI_EUNSUPPORTED,
                 "%s: f_src and add must be 16-byte aligned", who);
    MESO_REQUIRE(Ns <= 0x7fffffff && Nd <= 0x7fffffff, MESORASI_EUNSUPPORTED, "%s: size", who);
    const RrInterp ip{nit, dist, f_src, ld_src, Nd, Ns, add, ld_add, relu ? 1 : 0};
    return run_rr_mlp(nullptr, C, 0, nullptr, 0, 0, B * Nd, n_layers, dims, W, bias, relu_mask, y, ld_y,
                      as_stream(stream), &ip);
}

extern "C" size_t mesorasi_conventional_workspace(int64_t B, int64_t M, int32_t K, int32_t n_layers,
                                                  const int32_t* dims, int32_t dtype) {
    if (B < 0 || M < 0 || K < 1) return 0;
    const int64_t rows = B * M * K;
    if (check_mlp_spec("mesorasi_conventional_workspace", rows, n_layers, dims, dtype) != MESORASI_OK) return 0;
    return align256((size_t)rows * (size_t)dims[0] * 4) + mlp_ws_bytes(rows, n_layers, dims, dtype, true);
}

extern "C" int mesorasi_conventional_module(const float* xyz, const float* feat, int32_t cf, int64_t ld_f,
                                            const float* cxyz, const int32_t* nit, int64_t B, int64_t N, int64_t M,
                                            int32_t K, int32_t grouping, int32_t n_layers, const int32_t* dims,
                                            const void* const* W, const float* const* bias, uint32_t relu_mask,
                                            int32_t dtype, float* out, int64_t ld_out, void* ws, size_t ws_bytes,
                                            void* stream) {
    const char* who = "mesorasi_conventional_module";
    MESO_REQUIRE(B >= 0 && N >= 0 && M >= 0, MESORASI_EINVAL, "%s: negative size", who);
    MESO_REQUIRE(K >= 1, MESORASI_EINVAL, "%s: K = %d < 1", who, K);
    MESO_REQUIRE(grouping == 0 || grouping == 1, MESORASI_EINVAL, "%s: grouping = %d", who, grouping);
    MESO_REQUIRE(cf >= 0, MESORASI_EINVAL, "%s: cf < 0", who);
    const int64_t rows = B * M * K;
    int rc = check_mlp_spec(who, rows, n_layers, dims, dtype);
    if (rc != MESORASI_OK) return rc;
    const int cin = grouping == 0 ? 3 + cf : 2 * cf;
    MESO_REQUIRE(dims[0] == cin, MESORASI_EINVAL, "%s: dims[0] = %d, expected %d", who, dims[0], cin);
    MESO_REQUIRE(ld_out >= dims[n_layers], MESORASI_EINVAL, "%s: ld_out < dims[n_layers]", who);
    MESO_REQUIRE(cf == 0 || ld_f >= cf, MESORASI_EINVAL, "%s: ld_f < cf", who);
    MESO_REQUIRE(grouping == 0 || (cf >= 1 && M == N), MESORASI_EINVAL, "%s: edge grouping needs cf >= 1 and M == N",
                 who);
    MESO_REQUIRE((relu_mask >> (n_layers - 1)) & 1u, MESORASI_EUNSUPPORTED, "%s: the last layer needs ReLU", who);
    if (B == 0 || M == 0) return MESORASI_OK;
    MESO_REQUIRE(N >= 1, MESORASI_EINVAL, "%s: N = 0 with M > 0", who);
    MESO_REQUIRE(nit && out && W, MESORASI_EINVAL, "%s: NULL nit, out or W", who);
    if (grouping == 0) MESO_REQUIRE(xyz && cxyz && (cf == 0 || feat), MESORASI_EINVAL, "%s: NULL xyz/cxyz/feat", who);
    else MESO_REQUIRE(feat != nullptr, MESORASI_EINVAL, "%s: NULL feat", who);
    for (int l = 0; l < n_layers; ++l) MESO_REQUIRE(W[l] != nullptr, MESORASI_EINVAL, "%s: W[%d] is NULL", who, l);
    const size_t nfm_bytes = align256((size_t)rows * (size_t)cin * 4);
    const size_t need = nfm_bytes + mlp_ws_bytes(rows, n_layers, dims, dtype, true);
    MESO_REQUIRE(ws && ws_bytes >= need, MESORASI_EWORKSPACE, "%s: workspace %zu < %zu bytes", who, ws_bytes, need);
    MESO_REQUIRE(N <= 0x7fffffff && M <= 0x7fffffff, MESORASI_EUNSUPPORTED, "%s: size", who);
    hipStream_t s = as_stream(stream);
    if (grouping == 0 && dtype == MESORASI_F32) {
        // gather -> MLP -> max without the neighbor matrix: the fused kernel
        // (every layer narrow) or a split first layer that reads its rows
        // through nit
        GemmArgs a0{};
        a0.x1 = feat; a0.ld1 = ld_f; a0.c0 = 3; a0.c1 = cf; a0.W = W[0];
        if (fused_mlp_supported(n_layers, dims, dtype) || split_ok(a0, false)) {
            const MlpGather g{nit, M * K, N, K, cxyz};
            return run_mlp(xyz, 3, 3, cf > 0 ? feat : nullptr, cf, cf > 0 ? ld_f : 0, rows, n_layers, dims, W, bias,
                           relu_mask, dtype, MESORASI_F32, out, ld_out, K, static_cast<char*>(ws) + nfm_bytes, s, true,
                           &g);
        }
    }
    float* nfm = static_cast<float*>(ws);
    const int64_t blocks = std::min<int64_t>(ceil_div(rows * cin, 256), 16384);
    if (grouping == 0)
        group_pointnet_kernel<<<dim3((unsigned)blocks), dim3(256), 0, s>>>(xyz, feat, cf, ld_f, cxyz, nit, (int)N,
                                                                           (int)M, K, rows, nfm);
    else
        group_edge_kernel<<<dim3((unsigned)blocks), dim3(256), 0, s>>>(feat, cf, ld_f, nit, (int)N, K, rows, nfm);
    rc = after_launch(who);
    if (rc != MESORASI_OK) return rc;
    return run_mlp(nfm, cin, cin, nullptr, 0, 0, rows, n_layers, dims, W, bias, relu_mask, dtype, MESORASI_F32, out,
                   ld_out, K, static_cast<char*>(ws) + nfm_bytes, s, true);
}

extern "C" size_t mesorasi_ltd_workspace(int64_t B, int64_t M, int32_t K, int32_t n_layers, const int32_t* dims,
                                         int32_t dtype) {
    if (B < 0 || M < 0 || K < 1 || n_layers < 1) return 0;
    const int64_t rows = B * M * K;
    if (check_mlp_spec("mesorasi_ltd_workspace", rows, n_layers, dims, dtype) != MESORASI_OK) return 0;
    return align256((size_t)rows * (size_t)dims[0] * 4) + mlp_ws_bytes(rows, n_layers, dims, dtype, true);
}

extern "C" int mesorasi_ltd_module(const float* p1, int64_t ld_p, const float* q, int64_t ld_q, const float* b1,
                                   const int32_t* nit, int64_t B, int64_t N, int64_t M, int32_t K, int32_t C1,
                                   int32_t n_layers, const int32_t* dims, const void* const* W,
                                   const float* const* bias, uint32_t relu_mask, int32_t dtype, float* out,
                                   int64_t ld_out, void* ws, size_t ws_bytes, void* stream) {
    const char* who = "mesorasi_ltd_module";
    MESO_REQUIRE(B >= 0 && N >= 0 && M >= 0, MESORASI_EINVAL, "%s: negative size", who);
    MESO_REQUIRE(K >= 1 && C1 >= 1, MESORASI_EINVAL, "%s: K = %d, C1 = %d", who, K, C1);
    MESO_REQUIRE(n_layers >= 1, MESORASI_EUNSUPPORTED,
                 "%s: n_layers = %d; a one-layer module's limited order is its delayed order", who, n_layers);
    const int64_t rows = B * M * K;
    int rc = check_mlp_spec(who, rows, n_layers, dims, dtype);
    if (rc != MESORASI_OK) return rc;
    MESO_REQUIRE(dims[0] == C1, MESORASI_EINVAL, "%s: dims[0] = %d != C1 = %d", who, dims[0], C1);
    MESO_REQUIRE(ld_p >= C1 && ld_q >= C1, MESORASI_EINVAL, "%s: ld_p / ld_q < C1", who);
    MESO_REQUIRE(ld_out >= dims[n_layers], MESORASI_EINVAL, "%s: ld_out < dims[n_layers]", who);
    MESO_REQUIRE((relu_mask >> (n_layers - 1)) & 1u, MESORASI_EUNSUPPORTED, "%s: the last layer needs ReLU", who);
    if (B == 0 || M == 0) return MESORASI_OK;
    MESO_REQUIRE(N >= 1, MESORASI_EINVAL, "%s: N = 0 with M > 0", who);
    MESO_REQUIRE(p1 && q && nit && out && W, MESORASI_EINVAL, "%s: NULL p1, q, nit, out or W", who);
    for (int l = 0; l < n_layers; ++l) MESO_REQUIRE(W[l] != nullptr, MESORASI_EINVAL, "%s: W[%d] is NULL", who, l);
    const size_t h1_bytes = align256((size_t)rows * (size_t)C1 * 4);
    const size_t need = h1_bytes + mlp_ws_bytes(rows, n_layers, dims, dtype, true);
    MESO_REQUIRE(ws && ws_bytes >= need, MESORASI_EWORKSPACE, "%s: workspace %zu < %zu bytes", who, ws_bytes, need);
    MESO_REQUIRE(N <= 0x7fffffff && M <= 0x7fffffff, MESORASI_EUNSUPPORTED, "%s: size", who);
    hipStream_t s = as_stream(stream);
    const bool vec = C1 % 4 == 0 && ld_p % 4 == 0 && ld_q % 4 == 0 && aligned(p1, 16) && aligned(q, 16) &&
                     (b1 == nullptr || aligned(b1, 16));
    if (dtype == MESORASI_F32 &&
        (fused_mlp_supported(n_layers, dims, dtype) || (vec && aligned(W[0], 16)))) {
        // the first-layer rows ReLU(p1[j] - q[c] + b1) are formed in the next
        // layer's loader (fused kernel or gathered GEMM), never in memory
        const MlpGather g{nit, M * K, N, K, nullptr, q, ld_q, b1};
        return run_mlp(p1, C1, ld_p, nullptr, 0, 0, rows, n_layers, dims, W, bias, relu_mask, dtype, MESORASI_F32,
                       out, ld_out, K, static_cast<char*>(ws) + h1_bytes, s, true, &g);
    }
    float* h1 = static_cast<float*>(ws);
    const int64_t work = rows * (vec ? C1 / 4 : C1);
    const int64_t blocks = std::min<int64_t>(ceil_div(work, 256), 16384);
    if (vec)
        ltd_group_kernel<true><<<dim3((unsigned)blocks), dim3(256), 0, s>>>(p1, ld_p, q, ld_q, b1, nit, (int)N, (int)M,
                                                                           K, C1, rows, h1);
    else
        ltd_group_kernel<false><<<dim3((unsigned)blocks), dim3(256), 0, s>>>(p1, ld_p, q, ld_q, b1, nit, (int)N,
                                                                            (int)M, K, C1, rows, h1);
    rc = after_launch(who);
    if (rc != MESORASI_OK) return rc;
    return run_mlp(h1, C1, C1, nullptr, 0, 0, rows, n_layers, dims, W, bias, relu_mask, dtype, MESORASI_F32, out,
                   ld_out, K, static_cast<char*>(ws) + h1_bytes, s, true);
}

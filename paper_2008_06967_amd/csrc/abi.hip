// Library-wide pieces of the C ABI: status strings, thread-local error text,
// and the small element-wise entry points (bf16 cast, EdgeConv weight fold,
// zero fill used before pooled atomics).
#include <stdarg.h>
#include <stdio.h>

#include <cmath>

#include "common.h"

namespace meso {

static thread_local char g_last_error[512] = "";

int set_error(int status, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
    va_end(ap);
    return status;
}

int after_launch(const char* what) {
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return set_error(MESORASI_EHIP, "%s: kernel launch failed: %s", what, hipGetErrorString(e));
    return MESORASI_OK;
}

__global__ void zero_rows_kernel(float* __restrict__ y, int64_t rows, int64_t cols, int64_t ld) {
    const int64_t n = rows * cols;
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < n; e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t r = e / cols, c = e - r * cols;
        y[r * ld + c] = 0.0f;
    }
}

int zero_rows_f32(float* y, int64_t rows, int64_t cols, int64_t ld, hipStream_t s) {
    if (rows <= 0 || cols <= 0) return MESORASI_OK;
    const int64_t n = rows * cols;
    const int64_t blocks = std::min<int64_t>(ceil_div(n, 256), 4096);
    zero_rows_kernel<<<dim3((unsigned)blocks), dim3(256), 0, s>>>(y, rows, cols, ld);
    return after_launch("zero_rows");
}

__global__ void cast_bf16_kernel(const float* __restrict__ x, int64_t n, uint16_t* __restrict__ y) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        y[i] = f32_to_bf16(x[i]);
}

__global__ void edgeconv_fold_kernel(const float* __restrict__ W, const float* __restrict__ b, int C, int Cout,
                                     float* __restrict__ Wo, float* __restrict__ bo) {
    const int64_t n = (int64_t)Cout * C;
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < n; e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t o = e / C, c = e - o * C;
        const float w1 = W[o * 2 * C + c];
        const float w2 = W[o * 2 * C + C + c];
        Wo[o * C + c] = w1 - w2;
        Wo[(Cout + o) * C + c] = w2;
    }
    for (int64_t o = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; o < Cout; o += (int64_t)gridDim.x * blockDim.x) {
        bo[o] = b ? b[o] : 0.0f;
        bo[Cout + o] = 0.0f;
    }
}

// Entries of idx outside [0, bound): one atomic per wave (ballot count).
__global__ void count_out_of_range_kernel(const int32_t* __restrict__ idx, int64_t n, int32_t bound,
                                          int32_t* __restrict__ count) {
    for (int64_t i0 = blockIdx.x * (int64_t)blockDim.x; i0 < n; i0 += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = i0 + threadIdx.x;
        const bool bad = i < n && (idx[i] < 0 || idx[i] >= bound);
        const uint64_t m = ballot(bad);
        if ((threadIdx.x & 63) == 0 && m) atomicAdd(count, (int32_t)__builtin_popcountll(m));
    }
}

__global__ void zero_i32_kernel(int32_t* p) { *p = 0; }

}  // namespace meso

using namespace meso;

extern "C" int mesorasi_version(void) { return MESORASI_VERSION; }

extern "C" const char* mesorasi_strerror(int status) {
    switch (status) {
        case MESORASI_OK: return "ok";
        case MESORASI_EINVAL: return "invalid argument";
        case MESORASI_EUNSUPPORTED: return "unsupported argument";
        case MESORASI_EHIP: return "HIP runtime error";
        case MESORASI_EWORKSPACE: return "workspace too small";
        default: return "unknown status";
    }
}

extern "C" const char* mesorasi_last_error(void) { return g_last_error; }

extern "C" int mesorasi_cast_bf16(const float* x, int64_t n, uint16_t* y, void* stream) {
    MESO_REQUIRE(n >= 0, MESORASI_EINVAL, "mesorasi_cast_bf16: n = %lld < 0", (long long)n);
    if (n == 0) return MESORASI_OK;
    MESO_REQUIRE(x && y, MESORASI_EINVAL, "mesorasi_cast_bf16: NULL pointer");
    const int64_t blocks = std::min<int64_t>(ceil_div(n, 256), 8192);
    cast_bf16_kernel<<<dim3((unsigned)blocks), dim3(256), 0, as_stream(stream)>>>(x, n, y);
    return after_launch("mesorasi_cast_bf16");
}

extern "C" int mesorasi_edgeconv_fold(const float* W, const float* b, int32_t C, int32_t C_out, float* W_out,
                                      float* b_out, void* stream) {
    MESO_REQUIRE(W && W_out && b_out, MESORASI_EINVAL, "mesorasi_edgeconv_fold: NULL pointer");
    MESO_REQUIRE(C >= 1 && C_out >= 1, MESORASI_EINVAL, "mesorasi_edgeconv_fold: C = %d, C_out = %d", C, C_out);
    const int64_t n = (int64_t)C * C_out;
    const int64_t blocks = std::min<int64_t>(ceil_div(std::max<int64_t>(n, C_out), 256), 4096);
    edgeconv_fold_kernel<<<dim3((unsigned)blocks), dim3(256), 0, as_stream(stream)>>>(W, b, C, C_out, W_out, b_out);
    return after_launch("mesorasi_edgeconv_fold");
}

extern "C" int mesorasi_count_out_of_range(const int32_t* idx, int64_t n, int32_t bound, int32_t* count, void* stream) {
    MESO_REQUIRE(n >= 0, MESORASI_EINVAL, "mesorasi_count_out_of_range: n = %lld < 0", (long long)n);
    MESO_REQUIRE(count && (idx || n == 0), MESORASI_EINVAL, "mesorasi_count_out_of_range: NULL pointer");
    zero_i32_kernel<<<dim3(1), dim3(1), 0, as_stream(stream)>>>(count);
    int rc = after_launch("mesorasi_count_out_of_range");
    if (rc != MESORASI_OK || n == 0) return rc;
    const int64_t blocks = std::min<int64_t>(ceil_div(n, 256), 4096);
    count_out_of_range_kernel<<<dim3((unsigned)blocks), dim3(256), 0, as_stream(stream)>>>(idx, n, bound, count);
    return after_launch("mesorasi_count_out_of_range");
}

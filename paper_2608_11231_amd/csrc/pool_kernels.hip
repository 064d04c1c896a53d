// The cache keeps its per-block end states in bf16 (Sec. 4, environment):
// rounding a computed fp32 pool to that format, and moving the rows a batch
// needs from host memory into HBM ahead of the kernels that read them.
#include "pool_kernels.h"

namespace lkv {

// fp32 -> bf16, round to nearest even (the hardware conversion): eight elements
// per thread, 32-byte reads and 16-byte writes.  HBM-bound.
__global__ __launch_bounds__(256) void round_bf16_kernel(const float* __restrict__ src, bf16* __restrict__ dst,
                                                         int64_t n) {
    const int64_t n8 = n / 8;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t t0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    for (int64_t i = t0; i < n8; i += stride) {
        const f32x4 a = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(src) + 2 * i);
        const f32x4 b = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(src) + 2 * i + 1);
        bf16x8 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            o[e] = (bf16)a[e];
            o[4 + e] = (bf16)b[e];
        }
        reinterpret_cast<bf16x8*>(dst)[i] = o;
    }
    for (int64_t i = 8 * n8 + t0; i < n; i += stride) dst[i] = (bf16)src[i];
}

hipError_t launch_round_bf16(const float* src, void* dst, int64_t n, hipStream_t st) {
    int64_t blocks = (n / 8 + 255) / 256;
    if (blocks < 1) blocks = 1;
    if (blocks > 256 * 16) blocks = 256 * 16;
    hipLaunchKernelGGL(round_bf16_kernel, dim3((unsigned)blocks), dim3(256), 0, st, src,
                       reinterpret_cast<bf16*>(dst), n);
    return hipGetLastError();
}

hipError_t stage_rows(void* dst, const void* src, const int32_t* rows, int32_t n_rows, int64_t row_bytes,
                      hipStream_t st) {
    char* d = reinterpret_cast<char*>(dst);
    const char* s = reinterpret_cast<const char*>(src);
    int32_t i = 0;
    while (i < n_rows) {
        int32_t j = i + 1;
        while (j < n_rows && rows[j] == rows[j - 1] + 1) ++j;
        hipError_t e = hipMemcpyAsync(d + (int64_t)i * row_bytes, s + (int64_t)rows[i] * row_bytes,
                                      (size_t)(j - i) * row_bytes, hipMemcpyHostToDevice, st);
        if (e != hipSuccess) return e;
        i = j;
    }
    return hipSuccess;
}

}  // namespace lkv

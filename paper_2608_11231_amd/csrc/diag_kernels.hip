// Relative error of a constructed state against a reference state, per slice
// and per group of slices (Sec. 3.2's probe of the initial state against the
// full-prefix state, one number per layer).  HBM-bound: both states are read
// once; the squares are summed in fp64 (an fp32 x fp32 product is exact in
// fp64), in a fixed order, so results are reproducible run to run.
#include "diag_kernels.h"

namespace lkv {

namespace {

constexpr int RE_THREADS = 256;

__device__ __forceinline__ double wave_sum(double x) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m, 64);
    return x;
}

}  // namespace

// one workgroup per slice
__global__ __launch_bounds__(RE_THREADS) void rel_error_kernel(const float* __restrict__ S,
                                                               const float* __restrict__ R, int64_t slice_elems,
                                                               double* __restrict__ sq, double* __restrict__ rel) {
    __shared__ double part[2][RE_THREADS / 64];
    const int64_t s = blockIdx.x;
    const int tid = threadIdx.x;
    const f32x4* a = reinterpret_cast<const f32x4*>(S + s * slice_elems);
    const f32x4* b = reinterpret_cast<const f32x4*>(R + s * slice_elems);
    double num = 0.0, den = 0.0;
    for (int64_t i = tid; i < slice_elems / 4; i += RE_THREADS) {
        const f32x4 x = __builtin_nontemporal_load(a + i);
        const f32x4 y = __builtin_nontemporal_load(b + i);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const double d = (double)x[e] - (double)y[e];
            num += d * d;
            den += (double)y[e] * (double)y[e];
        }
    }
    num = wave_sum(num);
    den = wave_sum(den);
    if ((tid & 63) == 0) {
        part[0][tid >> 6] = num;
        part[1][tid >> 6] = den;
    }
    __syncthreads();
    if (tid == 0) {
        double n = 0.0, d = 0.0;
#pragma unroll
        for (int w = 0; w < RE_THREADS / 64; ++w) {
            n += part[0][w];
            d += part[1][w];
        }
        sq[2 * s] = n;
        sq[2 * s + 1] = d;
        rel[s] = sqrt(n) / sqrt(d);
    }
}

// one thread per group: the group's slices summed in slice order
__global__ __launch_bounds__(256) void rel_group_kernel(const double* __restrict__ sq, int32_t n_groups,
                                                        int32_t group, double* __restrict__ rel_group) {
    const int g = blockIdx.x * blockDim.x + threadIdx.x;
    if (g >= n_groups) return;
    double n = 0.0, d = 0.0;
    for (int i = 0; i < group; ++i) {
        n += sq[2 * ((int64_t)g * group + i)];
        d += sq[2 * ((int64_t)g * group + i) + 1];
    }
    rel_group[g] = sqrt(n) / sqrt(d);
}

hipError_t launch_rel_error(const float* S, const float* R, int32_t n_slices, int64_t slice_elems, int32_t group,
                            double* sq, double* rel, double* rel_group, hipStream_t st) {
    hipLaunchKernelGGL(rel_error_kernel, dim3(n_slices), dim3(RE_THREADS), 0, st, S, R, slice_elems, sq, rel);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || !rel_group) return e;
    const int32_t n_groups = n_slices / group;
    hipLaunchKernelGGL(rel_group_kernel, dim3((n_groups + 255) / 256), dim3(256), 0, st, sq, n_groups, group,
                       rel_group);
    return hipGetLastError();
}

}  // namespace lkv

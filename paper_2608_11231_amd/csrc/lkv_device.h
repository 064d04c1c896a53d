// Device-side building blocks shared by the lkv kernels (gfx950 / CDNA4).
//
// Matrix-core conventions used throughout.  A 16x16 fp32 accumulator tile
// ("acc tile") lives in one wave: lane l = 16*g + c holds column c and rows
// 4g..4g+3.  The bf16 MFMA instructions take their A operand with row = lane%16
// and their B operand with column = lane%16; the contraction index is spread
// over lane groups g and vector elements.  Because A and B map the contraction
// index identically, any bijection between "logical k" and (g, element) is a
// valid contraction.  The kernels use the one that makes an acc tile directly
// usable as a B operand: in each 16-wide slice of k, group g supplies logical
// k = 4g..4g+3 -- exactly the rows an acc tile already keeps in lane group g.
// A 32-wide MFMA therefore takes two 16-row acc tiles as its B operand, and
// its A operand is read from LDS as two 4-element runs per lane.
//
// One accumulation chain never mixes the 32-wide and the 16-wide MFMA: this
// compiler issues a dependent 16x16x16 right after a 16x16x32 on the same
// accumulator without wait states, and the 16-wide op then reads rows the
// wider op has not yet written.  An odd trailing 16-slice of a chain that
// started 32-wide is issued as a 32-wide op with a zero upper half.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lkv {

typedef __bf16 bf16;
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));

// 16x16 output, contraction over 32 (two 16-slices)
__device__ __forceinline__ f32x4 mma32(bf16x4 a0, bf16x4 a1, bf16x4 b0, bf16x4 b1, f32x4 c) {
    bf16x8 a = __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7);
    bf16x8 b = __builtin_shufflevector(b0, b1, 0, 1, 2, 3, 4, 5, 6, 7);
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// 16x16 output, contraction over one 16-slice
__device__ __forceinline__ f32x4 mma16(bf16x4 a, bf16x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(i16x4, a),
                                                      __builtin_bit_cast(i16x4, b), c, 0, 0, 0);
}

__device__ __forceinline__ f32x4 zero4() { return f32x4{0.f, 0.f, 0.f, 0.f}; }
__device__ __forceinline__ bf16x4 zero_bf16x4() { return bf16x4{(bf16)0.f, (bf16)0.f, (bf16)0.f, (bf16)0.f}; }

// round-to-nearest-even fp32 -> bf16
__device__ __forceinline__ bf16x4 to_bf16(f32x4 x) {
    return bf16x4{(bf16)x[0], (bf16)x[1], (bf16)x[2], (bf16)x[3]};
}
__device__ __forceinline__ f32x4 to_f32(bf16x4 x) {
    return f32x4{(float)x[0], (float)x[1], (float)x[2], (float)x[3]};
}

// x = hi + lo with hi = bf16(x) and lo = bf16(x - hi); x - hi is exact in fp32,
// so hi + lo carries 16 significant bits of x.
struct Split4 {
    bf16x4 hi, lo;
};
__device__ __forceinline__ Split4 split4(f32x4 x) {
    Split4 s;
    s.hi = to_bf16(x);
    s.lo = to_bf16(x - to_f32(s.hi));
    return s;
}

// LDS loads of 4 consecutive elements (8 / 16 bytes)
__device__ __forceinline__ bf16x4 lds4(const bf16* p) { return *reinterpret_cast<const bf16x4*>(p); }
__device__ __forceinline__ f32x4 lds4f(const float* p) { return *reinterpret_cast<const f32x4*>(p); }

// Transposed fragment read (gfx950 ds_read_b64_tr_b16).  Within each group of
// 16 lanes the instruction takes the 16 four-element vectors the lanes address
// as one 64-element run and hands lane i every 16th element starting at i.  With
// lane i of group g addressing M[r0 + 4g + i/4][c0 + 4(i%4)] of a row-major
// bf16 LDS matrix M, lane (g, c) receives M[r0 + 4g + j][c0 + c], j = 0..3:
// the MFMA operand fragment of M^T (row c0 + c, contraction rows r0 + 4g + j)
// without a transposed copy of M.
typedef short lds_i16x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ bf16x4 lds4_tr(const bf16* M, int stride, int r0, int c0, int g, int c) {
    const bf16* a = M + (r0 + 4 * g + (c >> 2)) * stride + c0 + 4 * (c & 3);
    typedef __attribute__((address_space(3))) lds_i16x4 lds_ptr_t;
    const lds_i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_ptr_t*)(a));
    return __builtin_bit_cast(bf16x4, v);
}

// Inclusive prefix sum across the 64 lanes of a wave.
__device__ __forceinline__ float wave_incl_scan(float x, int lane) {
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        float y = __shfl_up(x, d, 64);
        if (lane >= d) x += y;
    }
    return x;
}

// Workgroup -> work-unit map that gives each XCD a contiguous range of units.
// The hardware deals workgroups round-robin over the 8 XCDs (b % 8); units
// that are adjacent in the caller's order (same head, same request) then share
// one XCD's L2.  The map is a bijection on [0, n).
__device__ __forceinline__ int xcd_unit(int b, int n) {
    const int q = n >> 3, r = n & 7, x = b & 7, i = b >> 3;
    return x * q + min(x, r) + i;
}

// Memory fence + instruction barrier for one wave's own LDS traffic: orders a
// wave's LDS writes before its later LDS reads of other lanes' data.
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

}  // namespace lkv

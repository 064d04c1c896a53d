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

#include <type_traits>

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

// the same with one or both operands as a single 8-element fragment (see kq_pos)
__device__ __forceinline__ f32x4 mma32(bf16x8 a, bf16x4 b0, bf16x4 b1, f32x4 c) {
    bf16x8 b = __builtin_shufflevector(b0, b1, 0, 1, 2, 3, 4, 5, 6, 7);
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mma32(bf16x4 a0, bf16x4 a1, bf16x8 b, f32x4 c) {
    bf16x8 a = __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7);
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mma32(bf16x8 a, bf16x8 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// 16x16 output, contraction over one 16-slice
__device__ __forceinline__ f32x4 mma16(bf16x4 a, bf16x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(i16x4, a),
                                                      __builtin_bit_cast(i16x4, b), c, 0, 0, 0);
}

__device__ __forceinline__ f32x4 zero4() { return f32x4{0.f, 0.f, 0.f, 0.f}; }

// f(integral_constant<int, I>) for I = B .. E-1, unrolled at compile time
template <int B, int E, class F>
__device__ __forceinline__ void static_for(F&& f) {
    if constexpr (B < E) {
        f(std::integral_constant<int, B>());
        static_for<B + 1, E>(f);
    }
}
__device__ __forceinline__ bf16x4 zero_bf16x4() { return bf16x4{(bf16)0.f, (bf16)0.f, (bf16)0.f, (bf16)0.f}; }

// round-to-nearest-even fp32 -> bf16, two values per conversion instruction
// (packed through 32-bit words, so the pairs survive vector shuffles)
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{a, b}, bf16x2));
}
__device__ __forceinline__ bf16x4 to_bf16(f32x4 x) {
    return __builtin_bit_cast(bf16x4, uint2{pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3])});
}
// exact bf16 -> fp32 from the packed bits (one shift or mask per value)
__device__ __forceinline__ f32x4 to_f32(bf16x4 x) {
    const uint2 b = __builtin_bit_cast(uint2, x);
    return f32x4{__builtin_bit_cast(float, b.x << 16), __builtin_bit_cast(float, b.x & 0xffff0000u),
                 __builtin_bit_cast(float, b.y << 16), __builtin_bit_cast(float, b.y & 0xffff0000u)};
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

// The same split with x - hi formed on the matrix core: one 16x16x32 product
// of the negated identity (A) with the acc tile's own hi parts (B, upper 16-slice
// zero), accumulated onto x.  Every product but one per output is an exact zero
// and x - hi is representable, so the result is bit-identical to split4 while
// the unpack and subtract of every value (two VALU instructions) become a
// quarter of an MFMA.  neg_eye: lane (g, c) holds -1 at element j when 4g + j
// == c (the contraction bijection above, first 16-slice), zero elsewhere.
__device__ __forceinline__ bf16x8 neg_eye(int g, int c) {
    bf16x8 e;
#pragma unroll
    for (int j = 0; j < 8; ++j) e[j] = (j < 4 && 4 * g + j == c) ? (bf16)-1.f : (bf16)0.f;
    return e;
}
__device__ __forceinline__ Split4 split4_mm(f32x4 x, bf16x8 negI) {
    Split4 s;
    s.hi = to_bf16(x);
    const bf16x8 b = __builtin_shufflevector(s.hi, bf16x4{(bf16)0.f, (bf16)0.f, (bf16)0.f, (bf16)0.f},
                                             0, 1, 2, 3, 4, 5, 6, 7);
    s.lo = to_bf16(__builtin_amdgcn_mfma_f32_16x16x32_bf16(negI, b, x, 0, 0, 0));
    return s;
}

// Two acc tiles split at once, for the common case where their parts feed a
// 32-wide product as its two 16-slices.  Both tiles' hi parts form one 8-element
// B operand, which is exactly that product's fragment; the first tile's x - hi
// takes the negated identity on the first 16-slice (neg_eye), the second's the
// same identity moved to the second slice (neg_eye_hi).  No operand needs zero
// padding or reassembly, and every value is bit-identical to split4.
__device__ __forceinline__ bf16x8 neg_eye_hi(int g, int c) {
    bf16x8 e;
#pragma unroll
    for (int j = 0; j < 8; ++j) e[j] = (j >= 4 && 4 * g + j - 4 == c) ? (bf16)-1.f : (bf16)0.f;
    return e;
}
struct Split8 {
    bf16x4 hi0, hi1, lo0, lo1;
};
__device__ __forceinline__ Split8 split8_mm(f32x4 x0, f32x4 x1, bf16x8 negI, bf16x8 negIh) {
    const bf16x8 hi = __builtin_shufflevector(to_bf16(x0), to_bf16(x1), 0, 1, 2, 3, 4, 5, 6, 7);
    const bf16x4 l0 = to_bf16(__builtin_amdgcn_mfma_f32_16x16x32_bf16(negI, hi, x0, 0, 0, 0));
    const bf16x4 l1 = to_bf16(__builtin_amdgcn_mfma_f32_16x16x32_bf16(negIh, hi, x1, 0, 0, 0));
    Split8 s;
    s.hi0 = __builtin_shufflevector(hi, hi, 0, 1, 2, 3);
    s.hi1 = __builtin_shufflevector(hi, hi, 4, 5, 6, 7);
    s.lo0 = l0;
    s.lo1 = l1;
    return s;
}

// LDS loads of 4 / 8 consecutive elements (8 / 16 / 16 bytes)
__device__ __forceinline__ bf16x4 lds4(const bf16* p) { return *reinterpret_cast<const bf16x4*>(p); }
__device__ __forceinline__ bf16x8 lds8(const bf16* p) { return *reinterpret_cast<const bf16x8*>(p); }

// Column order of token-major K / Q tiles in LDS.  A 32-wide product needs, in
// lane group g, the elements 4g..4g+3 and 16+4g..16+4g+3 of each 32-column slice
// (the contraction bijection above).  Rows are stored with those two runs side
// by side at 8g..8g+7, so one 16-byte read fetches a whole fragment; every
// aligned run of 4 columns stays contiguous, so transposed reads still work.
// Tiles only 16 columns wide keep the natural order.
template <int DK>
__device__ __forceinline__ constexpr int kq_pos(int d) {
    return DK >= 32 ? ((d & ~31) | ((d & 12) << 1) | ((d & 16) >> 2) | (d & 3)) : d;
}
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

// lds4_tr for a K / Q tile stored in kq_pos order: column block c0 (a multiple of 16).
template <int DK>
__device__ __forceinline__ bf16x4 lds4_tr_kq(const bf16* M, int stride, int r0, int c0, int g, int c) {
    const bf16* a = M + (r0 + 4 * g + (c >> 2)) * stride + kq_pos<DK>(c0 + 4 * (c & 3));
    typedef __attribute__((address_space(3))) lds_i16x4 lds_ptr_t;
    const lds_i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_ptr_t*)(a));
    return __builtin_bit_cast(bf16x4, v);
}

// Inclusive prefix sum across the 64 lanes of a wave, in registers: shifts by
// 1, 2, 4, 8 within each row of 16 lanes (DPP row_shr, zero-filled), then the
// row totals are carried forward with DPP row_bcast:15 (into rows 1 and 3) and
// row_bcast:31 (into rows 2 and 3).
template <int CTRL, int ROW_MASK, bool BOUND_ZERO>
__device__ __forceinline__ float dpp_mov(float x) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, ROW_MASK, 0xf,
                                                                 BOUND_ZERO));
}
__device__ __forceinline__ float wave_incl_scan(float x) {
    x += dpp_mov<0x111, 0xf, true>(x);  // row_shr:1
    x += dpp_mov<0x112, 0xf, true>(x);  // row_shr:2
    x += dpp_mov<0x114, 0xf, true>(x);  // row_shr:4
    x += dpp_mov<0x118, 0xf, true>(x);  // row_shr:8
    x += dpp_mov<0x142, 0xa, false>(x);  // row_bcast:15 -> rows 1, 3
    x += dpp_mov<0x143, 0xc, false>(x);  // row_bcast:31 -> rows 2, 3
    return x;
}

// Workgroup -> work-unit map that gives each XCD a contiguous range of units.
// The hardware deals workgroups round-robin over the 8 XCDs (b % 8); units
// that are adjacent in the caller's order then share one XCD's L2 (callers
// order their units so that adjacent ones read the same rows).  The map is a
// bijection on [0, n).
__device__ __forceinline__ int xcd_unit(int b, int n) {
    const int q = n >> 3, r = n & 7, x = b & 7, i = b >> 3;
    return x * q + min(x, r) + i;
}

// Workgroup barrier for LDS traffic: waits for this wave's LDS operations only,
// so global loads issued before it stay in flight across it (a __syncthreads
// would also drain them).  Only for barriers that order LDS accesses.
__device__ __forceinline__ void lds_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Memory fence + instruction barrier for one wave's own LDS traffic: orders a
// wave's LDS writes before its later LDS reads of other lanes' data.
// Point-to-point signal between waves of one workgroup through an LDS counter,
// for producers and a consumer inside one barrier interval.  lds_signal: after
// this wave's earlier LDS writes have completed, lane 0 adds 1 (the LDS executes
// its operations in order, so a wave that reads the new count and then reads
// those locations sees the writes).  lds_wait_count: polls (with s_sleep) until
// the count reaches `target`, at most `limit` times, and returns whether it did.
// A legitimate wait is a fraction of a chunk (well under 200 polls); the default
// bound of 2^14 polls (about a millisecond) makes a missing signal end the wait
// within milliseconds, never in a workgroup that stays resident.  The caller
// turns a wait that gave up into NaN results; limit 0 never polls and always
// gives up.
__device__ __forceinline__ void lds_signal(uint32_t* cnt, int lane) {
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    if (lane == 0) __hip_atomic_fetch_add(cnt, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ bool lds_wait_count(const uint32_t* cnt, uint32_t target, int limit) {
    bool reached = false;
    for (int spin = 0; spin < limit; ++spin) {
        const uint32_t v = __hip_atomic_load(cnt, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        if (__builtin_amdgcn_readfirstlane(v) >= target) {
            reached = true;
            break;
        }
        __builtin_amdgcn_s_sleep(1);
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    return reached;
}

__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

}  // namespace lkv

// Decode step: one token per request advances the state by one step of the
// recurrence (Eq. 1 with Eq. 3 / Eq. 2) and produces that token's output.
// This is what follows the online prefill: the final state it keeps is the
// only thing decoding needs.
//
// Memory-bound: every state element is read and written once.  A workgroup is
// one wave that owns a few rows of one (request, head) state (8, or the 16
// rows one instruction covers at dk = 16: more, smaller waves keep more of
// HBM busy; 8 rows measured 5% faster than 16 and 4 rows slower); the DK/4
// lanes of a row hold four consecutive columns each, so a row is one
// coalesced 16-byte access per lane and the row's dot products are
// reductions over DK/4 lanes.
#include "decode_kernels.h"

namespace lkv {

namespace {

// element i of a packed row of bf16 / fp32 values, widened to fp32
__device__ __forceinline__ f32x4 load4(const void* base, int64_t elem, bool bf) {
    if (bf) {
        const uint2 u = *reinterpret_cast<const uint2*>(reinterpret_cast<const uint16_t*>(base) + elem);
        return f32x4{__builtin_bit_cast(float, u.x << 16), __builtin_bit_cast(float, u.x & 0xffff0000u),
                     __builtin_bit_cast(float, u.y << 16), __builtin_bit_cast(float, u.y & 0xffff0000u)};
    }
    return *reinterpret_cast<const f32x4*>(reinterpret_cast<const float*>(base) + elem);
}
__device__ __forceinline__ float load1(const void* base, int64_t elem, bool bf) {
    if (bf) return __builtin_bit_cast(float, (uint32_t)reinterpret_cast<const uint16_t*>(base)[elem] << 16);
    return reinterpret_cast<const float*>(base)[elem];
}
__device__ __forceinline__ void store1(void* base, int64_t elem, float x, bool bf) {
    if (bf) reinterpret_cast<bf16*>(base)[elem] = (bf16)x;  // round to nearest even
    else reinterpret_cast<float*>(base)[elem] = x;
}

// sum over the L lanes of a row group (L a power of two, groups aligned)
template <int L>
__device__ __forceinline__ float group_sum(float x) {
#pragma unroll
    for (int m = 1; m < L; m <<= 1) x += __shfl_xor(x, m, 64);
    return x;
}

}  // namespace

// state rows per wave
__host__ __device__ constexpr int decode_rows(int dk) { return 256 / dk > 8 ? 256 / dk : 8; }

template <int DK, int FAM>
__global__ __launch_bounds__(64) void decode_kernel(DecodeArgs p) {
    constexpr int LPR = DK / 4;        // lanes per row
    constexpr int RPI = 64 / LPR;      // rows per wave instruction
    constexpr int ROWS = decode_rows(DK);
    constexpr int IT = ROWS / RPI;     // iterations over the wave's rows
    static_assert(IT >= 1 && ROWS % RPI == 0, "rows per wave");
    const int lane = threadIdx.x;
    const int c4 = lane % LPR, rsub = lane / LPR;
    const int tiles = p.dv / ROWS;
    const int tile = blockIdx.x % tiles;
    const int h = (blockIdx.x / tiles) % p.h_v;
    const int r = blockIdx.x / (tiles * p.h_v);
    const int hq = h / (p.h_v / p.h_qk);
    const bool bf = p.io_bf16 != 0;

    const int64_t qk_elem = ((int64_t)r * p.h_qk + hq) * DK + 4 * c4;
    const f32x4 k4 = load4(p.k, qk_elem, bf);
    const f32x4 q4 = load4(p.q, qk_elem, bf);
    const int64_t gh = (int64_t)r * p.h_v + h;
    float decay, coef;  // S <- decay * S + coef * (...)
    if (FAM == 0) {
        decay = __expf(load1(p.g, gh, p.gate_bf16 != 0));
        coef = load1(p.beta, gh, p.gate_bf16 != 0);
    } else {
        const float dt = reinterpret_cast<const float*>(p.g)[gh];
        decay = __expf(dt * p.A[h]);
        coef = dt;
    }
    float* S = p.S + (gh * p.dv + ROWS * tile) * DK + 4 * c4;
    const int64_t v0 = gh * p.dv + ROWS * tile;

    f32x4 s[IT];
    float vr[IT];
#pragma unroll
    for (int i = 0; i < IT; ++i) {
        const int row = RPI * i + rsub;
        s[i] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(S + (int64_t)row * DK));
        vr[i] = load1(p.v, v0 + row, bf);
    }
#pragma unroll
    for (int i = 0; i < IT; ++i) {
        const int row = RPI * i + rsub;
        f32x4 sn;
        if (FAM == 0) {
            // delta rule: S <- alpha S + beta (v - alpha S k) k^T
            const float kv = group_sum<LPR>(s[i][0] * k4[0] + s[i][1] * k4[1] + s[i][2] * k4[2] + s[i][3] * k4[3]);
            const float d = coef * (vr[i] - decay * kv);
            sn = decay * s[i] + d * k4;
        } else {
            // S <- exp(dt A) S + dt x B^T
            sn = decay * s[i] + (coef * vr[i]) * k4;
        }
        __builtin_nontemporal_store(sn, reinterpret_cast<f32x4*>(S + (int64_t)row * DK));
        const float o = group_sum<LPR>(sn[0] * q4[0] + sn[1] * q4[1] + sn[2] * q4[2] + sn[3] * q4[3]);
        if (c4 == 0 && p.out) store1(p.out, v0 + row, (FAM == 0 ? p.scale : 1.f) * o, bf);
    }
}

template <int FAM>
static hipError_t launch_decode_f(int dk, const DecodeArgs& a, hipStream_t st) {
    const int64_t grid = (int64_t)a.n_req * a.h_v * (a.dv / decode_rows(dk));
    switch (dk) {
        case 16: hipLaunchKernelGGL((decode_kernel<16, FAM>), dim3(grid), dim3(64), 0, st, a); break;
        case 32: hipLaunchKernelGGL((decode_kernel<32, FAM>), dim3(grid), dim3(64), 0, st, a); break;
        case 64: hipLaunchKernelGGL((decode_kernel<64, FAM>), dim3(grid), dim3(64), 0, st, a); break;
        case 128: hipLaunchKernelGGL((decode_kernel<128, FAM>), dim3(grid), dim3(64), 0, st, a); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_decode(int family, int dk, const DecodeArgs& a, hipStream_t st) {
    return family == 0 ? launch_decode_f<0>(dk, a, st) : launch_decode_f<1>(dk, a, st);
}

}  // namespace lkv

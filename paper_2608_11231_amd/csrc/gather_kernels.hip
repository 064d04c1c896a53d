// Selected-position gather: the recompute step advances each recurrent state
// through the selected positions only, in context order (Alg. 1, selection
// and recompute), so its token stream is the context's rows at those
// positions.  Pure data movement, bit-exact.
//
// One workgroup copies one selected token: its q, k and v rows in 16-byte
// units (rows of dk or dv elements are multiples of 16 bytes) and its h_v
// gate values.  HBM-bound: each byte is read once and written once.  The
// work before the copy is a few dependent index loads, so they are kept
// short: the token's position is requested first, the request is found with
// one parallel pass over the selection offsets (a count, not a binary search
// of dependent loads), and every array's loads are issued before any store.
#include "gather_kernels.h"

namespace lkv {

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ int64_t clamp64(int64_t x, int64_t hi) { return x < 0 ? 0 : (x > hi ? hi : x); }

constexpr int GT = 256;  // threads per workgroup
constexpr int UPT = 4;   // 16-byte units per thread and array held in registers

}  // namespace

__global__ __launch_bounds__(GT) void gather_kernel(GatherArgs p) {
    const int64_t j = blockIdx.x;
    const int tid = threadIdx.x;
    __shared__ int64_t s_cu[GT + 1];
    const int64_t ps = p.pos[j];  // independent of the request: requested first
    // The request r holding selected row j: with clamped offsets cu[0..n_req]
    // non-decreasing, r + 1 = #{t : cu[t] <= j}.  Each thread tests one offset
    // (in passes of GT for very many requests); the answer is then checked,
    // cu[r] <= j < cu[r+1], so offsets outside the contract still give an
    // in-range answer or the NaN row, never an out-of-range read.
    int cnt = 0;
    for (int t0 = 0; t0 <= p.n_req; t0 += GT) {
        const int t = t0 + tid;
        const int64_t c = t <= p.n_req ? clamp64(p.sel_cu[t], p.n_sel) : INT64_MAX;
        if (t0 == 0) s_cu[tid] = c;
        cnt += __syncthreads_count(c <= j);
    }
    const int r = cnt - 1;
    int64_t src_row = -1;
    if (r >= 0 && r < p.n_req) {
        const int64_t lo = r < GT ? s_cu[r] : clamp64(p.sel_cu[r], p.n_sel);
        const int64_t hi = r + 1 < GT ? s_cu[r + 1] : clamp64(p.sel_cu[r + 1], p.n_sel);
        if (lo <= j && j < hi) {
            const int64_t c0 = clamp64(p.ctx_cu[r], p.ctx_tok);
            const int64_t c1 = clamp64(p.ctx_cu[r + 1], p.ctx_tok);
            if (ps >= 0 && ps < c1 - c0) src_row = c0 + ps;
        }
    }
    if (src_row < 0) {
        // no valid source row: NaN of each array's dtype
#pragma unroll
        for (int a = 0; a < GATHER_ARRAYS; ++a) {
            if (!p.dst[a]) continue;
            const int rb = p.row_bytes[a];
            char* d = reinterpret_cast<char*>(p.dst[a]) + j * rb;
            const uint32_t nan = p.elem_bytes[a] == 2 ? 0x7fc07fc0u : 0x7fc00000u;
            for (int u = tid; u < rb / 2; u += GT)
                reinterpret_cast<uint16_t*>(d)[u] = (uint16_t)(nan >> (16 * (u & 1)));
        }
        return;
    }
    // 16-byte rows: the first GT * UPT units of every array, all loads first
    u32x4 v[GATHER_ARRAYS][UPT];
#pragma unroll
    for (int a = 0; a < GATHER_ARRAYS; ++a) {
        const int rb = p.row_bytes[a];
        if (!p.dst[a] || rb % 16) continue;
        const u32x4* s = reinterpret_cast<const u32x4*>(reinterpret_cast<const char*>(p.src[a]) + src_row * rb);
#pragma unroll
        for (int k = 0; k < UPT; ++k) {
            const int u = tid + k * GT;
            if (u < rb / 16) v[a][k] = __builtin_nontemporal_load(s + u);
        }
    }
#pragma unroll
    for (int a = 0; a < GATHER_ARRAYS; ++a) {
        const int rb = p.row_bytes[a];
        if (!p.dst[a] || rb % 16) continue;
        u32x4* d = reinterpret_cast<u32x4*>(reinterpret_cast<char*>(p.dst[a]) + j * rb);
#pragma unroll
        for (int k = 0; k < UPT; ++k) {
            const int u = tid + k * GT;
            if (u < rb / 16) d[u] = v[a][k];
        }
    }
    // the rest: units past GT * UPT, and rows that are not a multiple of 16 bytes
#pragma unroll
    for (int a = 0; a < GATHER_ARRAYS; ++a) {
        if (!p.dst[a]) continue;
        const int rb = p.row_bytes[a];
        char* d = reinterpret_cast<char*>(p.dst[a]) + j * rb;
        const char* s = reinterpret_cast<const char*>(p.src[a]) + src_row * rb;
        if (rb % 16 == 0) {
            for (int u = tid + GT * UPT; u < rb / 16; u += GT)
                reinterpret_cast<u32x4*>(d)[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(s) + u);
        } else if (rb % 4 == 0) {
            for (int u = tid; u < rb / 4; u += GT)
                reinterpret_cast<uint32_t*>(d)[u] = reinterpret_cast<const uint32_t*>(s)[u];
        } else {
            for (int u = tid; u < rb / 2; u += GT)
                reinterpret_cast<uint16_t*>(d)[u] = reinterpret_cast<const uint16_t*>(s)[u];
        }
    }
}

hipError_t launch_gather(const GatherArgs& a, hipStream_t st) {
    hipLaunchKernelGGL(gather_kernel, dim3((unsigned)a.n_sel), dim3(GT), 0, st, a);
    return hipGetLastError();
}

}  // namespace lkv

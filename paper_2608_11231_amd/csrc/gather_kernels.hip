// Selected-position gather: the recompute step advances each recurrent state
// through the selected positions only, in context order (Alg. 1, selection
// and recompute), so its token stream is the context's rows at those
// positions.  Pure data movement, bit-exact.
//
// One workgroup copies one selected token: its q, k and v rows in 16-byte
// units (rows of dk or dv elements are multiples of 16 bytes) and its h_v
// gate values element by element.  HBM-bound: each byte is read once and
// written once.
#include "gather_kernels.h"

namespace lkv {

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ int64_t clamp64(int64_t x, int64_t hi) { return x < 0 ? 0 : (x > hi ? hi : x); }

// the request that selected row j belongs to: the last r with cu[r] <= j
// (clamped offsets; empty segments are skipped), or -1 when there is none
__device__ int find_segment(const int32_t* cu, int n_req, int64_t n, int64_t j) {
    if (clamp64(cu[0], n) > j) return -1;
    int lo = 0, hi = n_req;  // cu[lo] <= j
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (clamp64(cu[mid], n) <= j) lo = mid;
        else hi = mid;
    }
    return clamp64(cu[lo + 1], n) > j ? lo : -1;
}

}  // namespace

__global__ __launch_bounds__(256) void gather_kernel(GatherArgs p) {
    const int64_t j = blockIdx.x;
    const int tid = threadIdx.x;
    const int r = find_segment(p.sel_cu, p.n_req, p.n_sel, j);
    int64_t src_row = -1;
    if (r >= 0) {
        const int64_t c0 = clamp64(p.ctx_cu[r], p.ctx_tok);
        const int64_t c1 = clamp64(p.ctx_cu[r + 1], p.ctx_tok);
        const int64_t ps = p.pos[j];
        if (ps >= 0 && ps < c1 - c0) src_row = c0 + ps;
    }
#pragma unroll
    for (int a = 0; a < GATHER_ARRAYS; ++a) {
        if (!p.dst[a]) continue;
        const int rb = p.row_bytes[a];
        char* d = reinterpret_cast<char*>(p.dst[a]) + j * rb;
        if (src_row < 0) {
            // no valid source row: NaN of the array's dtype
            const uint32_t nan = p.elem_bytes[a] == 2 ? 0x7fc07fc0u : 0x7fc00000u;
            for (int u = tid; u < rb / 2; u += 256)
                reinterpret_cast<uint16_t*>(d)[u] = (uint16_t)(nan >> (16 * (u & 1)));
            continue;
        }
        const char* s = reinterpret_cast<const char*>(p.src[a]) + src_row * rb;
        if (rb % 16 == 0) {
            for (int u = tid; u < rb / 16; u += 256)
                reinterpret_cast<u32x4*>(d)[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(s) + u);
        } else if (rb % 4 == 0) {
            for (int u = tid; u < rb / 4; u += 256)
                reinterpret_cast<uint32_t*>(d)[u] = reinterpret_cast<const uint32_t*>(s)[u];
        } else {
            for (int u = tid; u < rb / 2; u += 256)
                reinterpret_cast<uint16_t*>(d)[u] = reinterpret_cast<const uint16_t*>(s)[u];
        }
    }
}

hipError_t launch_gather(const GatherArgs& a, hipStream_t st) {
    hipLaunchKernelGGL(gather_kernel, dim3((unsigned)a.n_sel), dim3(256), 0, st, a);
    return hipGetLastError();
}

}  // namespace lkv

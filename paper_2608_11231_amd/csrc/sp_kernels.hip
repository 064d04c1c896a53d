// Set-up of the sequence-parallel chunk scan.  Each request's online stream
// [cu[r], cu[r+1]) is cut into `pieces` consecutive pieces whose lengths are
// whole chunks (the last one takes the remainder; trailing pieces may be
// empty).  The scan is then Eq. 5 applied piece after piece: every piece's
// (transition, state from zero) pair is independent, and the composition of
// the request's initial state with the pairs of pieces 0..p-1 (Eq. 6 from a
// non-empty prefix) is piece p's start state.
//
// This kernel writes the index arrays of that composition -- request r
// becomes the block list [initial-state row, piece r*P, ..., piece r*P+P-1],
// the initial-state row being pool row n_req*P + r -- and copies the requests'
// initial states (or zeros) into those pool rows.
#include "sp_kernels.h"

namespace lkv {

__global__ __launch_bounds__(256) void sp_setup_kernel(const int32_t* __restrict__ cu, int32_t n_req, int32_t P,
                                                       int32_t CH, int64_t n_tok, int32_t* __restrict__ piece_cu,
                                                       int32_t* __restrict__ blk_ids, int32_t* __restrict__ blk_cu,
                                                       const f32x4* __restrict__ S_init, f32x4* __restrict__ init_rows,
                                                       int64_t state4) {
    const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t rr = gid; rr < n_req; rr += stride) {
        const int32_t r = (int32_t)rr;
        int64_t t0 = cu[r], t1 = cu[r + 1];
        t0 = t0 < 0 ? 0 : (t0 > n_tok ? n_tok : t0);
        t1 = t1 < t0 ? t0 : (t1 > n_tok ? n_tok : t1);
        const int64_t len = t1 - t0;
        const int64_t per = ((len + P - 1) / P + CH - 1) / CH * CH;  // whole chunks per piece
        for (int32_t p = 0; p < P; ++p) {
            const int64_t off = (int64_t)p * per;
            piece_cu[(int64_t)r * P + p] = (int32_t)(t0 + (off < len ? off : len));
        }
        if (r == n_req - 1) piece_cu[(int64_t)n_req * P] = (int32_t)t1;
        const int64_t k0 = (int64_t)r * (P + 1);
        blk_cu[r] = (int32_t)k0;
        if (r == n_req - 1) blk_cu[n_req] = (int32_t)(k0 + P + 1);
        blk_ids[k0] = n_req * P + r;
        for (int32_t p = 0; p < P; ++p) blk_ids[k0 + 1 + p] = r * P + p;
    }
    const int64_t total = (int64_t)n_req * state4;
    for (int64_t i = gid; i < total; i += stride)
        init_rows[i] = S_init ? S_init[i] : f32x4{0.f, 0.f, 0.f, 0.f};
}

hipError_t launch_sp_setup(const int32_t* cu, int32_t n_req, int32_t pieces, int32_t chunk, int64_t n_tok,
                           int32_t* piece_cu, int32_t* blk_ids, int32_t* blk_cu, const float* S_init,
                           float* init_rows, int64_t state_elems, hipStream_t st) {
    const int64_t total = (int64_t)n_req * (state_elems / 4);
    int64_t blocks = ((total > n_req ? total : n_req) + 255) / 256;
    if (blocks > 1024) blocks = 1024;
    hipLaunchKernelGGL(sp_setup_kernel, dim3((unsigned)blocks), dim3(256), 0, st, cu, n_req, pieces, chunk, n_tok,
                       piece_cu, blk_ids, blk_cu, reinterpret_cast<const f32x4*>(S_init),
                       reinterpret_cast<f32x4*>(init_rows), state_elems / 4);
    return hipGetLastError();
}

}  // namespace lkv

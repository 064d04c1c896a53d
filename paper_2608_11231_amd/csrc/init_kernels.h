// Host-side launchers of the state-initialisation kernels.
#pragma once
#include "lkv_device.h"

namespace lkv {

struct ComposeArgs {
    const void* B_pool;    // [n_blk,h_v,dv,dk] f32, or bf16 when bf16_pool
    const float* M_pool;   // [n_blk,h_v,dk,dk]
    const int32_t* blk_ids;
    const int32_t* blk_cu;
    int32_t n_ids, n_blk, h_v, dv;
    float* S;              // [n_req,h_v,dv,dk]
    float* S_steps;        // or null: the state after each block but a request's last,
                           // request r's block at position j going to row j - r
    int32_t tiles;         // row tiles over dv: 16*nw rows each, 64 for nw = 8
    int32_t nw;            // waves per workgroup: 1, 2, 4 (one 16-row tile each) or 8 (see the kernel)
    int32_t n_units;
    bool bf16_pool;
};

hipError_t launch_init_single(int32_t n_req, int32_t n_blk, int64_t per_req, const void* B_pool, bool bf16_pool,
                              const int32_t* src, float* S, hipStream_t st);
hipError_t launch_compose_ssd(int32_t n_req, int32_t n_blk, int32_t H, int64_t per_head, const void* B_pool,
                              bool bf16_pool, const float* Lam, const int32_t* ids, const int32_t* blk_cu,
                              int32_t n_ids, float* S, float* S_steps, hipStream_t st);
hipError_t launch_compose_gdn(int dk, const ComposeArgs& a, hipStream_t st);
hipError_t launch_ssd_lambda(const int32_t* cu, int32_t n_seq, int64_t n_tok, int32_t H, const float* dt,
                             const float* A, float* Lam, hipStream_t st);

}  // namespace lkv

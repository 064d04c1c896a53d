// Host-side launcher of the selected-position gather.
#pragma once
#include "lkv_device.h"

namespace lkv {

// The five per-token arrays of a token stream: q, k, v, g, beta.
constexpr int GATHER_ARRAYS = 5;

struct GatherArgs {
    const int32_t* ctx_cu;   // [n_req+1] context segments
    int64_t ctx_tok;         // context rows (clamp bound of ctx_cu)
    const int32_t* pos;      // [n_sel] position inside the request's context
    const int32_t* sel_cu;   // [n_req+1] selected segments
    int64_t n_sel;
    int32_t n_req;
    const void* src[GATHER_ARRAYS];
    void* dst[GATHER_ARRAYS];      // null: array not gathered
    int32_t row_bytes[GATHER_ARRAYS];
    int32_t elem_bytes[GATHER_ARRAYS];  // 2 (bf16) or 4 (f32): the NaN fill pattern
};

hipError_t launch_gather(const GatherArgs& a, hipStream_t st);

}  // namespace lkv

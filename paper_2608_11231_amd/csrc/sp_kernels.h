// Host-side launcher of the sequence-parallel scan's set-up kernel.
#pragma once
#include "lkv_device.h"

namespace lkv {

hipError_t launch_sp_setup(const int32_t* cu, int32_t n_req, int32_t pieces, int32_t chunk, int64_t n_tok,
                           int32_t* piece_cu, int32_t* blk_ids, int32_t* blk_cu, const float* S_init,
                           float* init_rows, int64_t state_elems, hipStream_t st);

}  // namespace lkv

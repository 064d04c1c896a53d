// Cached-state pool in the cache's bf16 storage format: rounding of a state
// pool to bf16 and host-to-device staging of pool rows.
#pragma once
#include "lkv_device.h"

namespace lkv {

hipError_t launch_round_bf16(const float* src, void* dst, int64_t n, hipStream_t st);

// dst row i <- src row rows[i] (rows of row_bytes bytes), as hipMemcpyAsync
// calls on `st`, one per run of consecutive source rows.
hipError_t stage_rows(void* dst, const void* src, const int32_t* rows, int32_t n_rows, int64_t row_bytes,
                      hipStream_t st);

}  // namespace lkv

// Instantiations of the chunk kernel: Mamba-2 (SSD), block-summary mode.
#include "chunk_kernel.h"

namespace lkv {

hipError_t launch_chunk_ssd_summary(int dk, int chunk, bool f32io, const ScanArgs& a, hipStream_t st) {
#define LKV_CASE(DK_, CH_)                                                                   \
    if (dk == DK_ && chunk == CH_) {                                                        \
        if (!f32io) return launch_chunk_s<FAM_SSD, DK_, CH_, false, true>(a, st);              \
        if constexpr (DK_ <= 64) return launch_chunk_s<FAM_SSD, DK_, CH_, true, true>(a, st);  \
        return hipErrorInvalidValue; /* fp32 q/k/v are supported up to dk = 64 */           \
    }
    LKV_CASE(16, 16) LKV_CASE(32, 16) LKV_CASE(64, 16) LKV_CASE(128, 16)
    LKV_CASE(16, 64) LKV_CASE(32, 64) LKV_CASE(64, 64) LKV_CASE(128, 64)
#undef LKV_CASE
    return hipErrorInvalidValue;
}

}  // namespace lkv

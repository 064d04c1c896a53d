// Instantiations of the chunk kernel: Gated DeltaNet, online scan with outputs.
#include "chunk_kernel.h"

namespace lkv {

hipError_t launch_chunk_gdn_scan(int dk, int chunk, bool f32io, const ScanArgs& a, hipStream_t st) {
#define LKV_CASE(DK_, CH_)                                                                   \
    if (dk == DK_ && chunk == CH_) {                                                        \
        if (!f32io) return launch_chunk_s<FAM_GDN, DK_, CH_, false, false>(a, st);              \
        if constexpr (DK_ <= 64) return launch_chunk_s<FAM_GDN, DK_, CH_, true, false>(a, st);  \
        return hipErrorInvalidValue; /* fp32 q/k/v are supported up to dk = 64 */           \
    }
    LKV_CASE(16, 16) LKV_CASE(32, 16) LKV_CASE(64, 16) LKV_CASE(128, 16)
    LKV_CASE(16, 64) LKV_CASE(32, 64) LKV_CASE(64, 64) LKV_CASE(128, 64)
#undef LKV_CASE
    return hipErrorInvalidValue;
}

}  // namespace lkv

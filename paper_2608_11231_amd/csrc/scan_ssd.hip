// Instantiations and dispatch of the chunkwise scan kernel for the
// Mamba-2 (SSD) family.
#include "scan_kernel.h"

namespace lkv {

#define LKV_CASE(DK_, CH_)                                                              \
    if (dk == DK_ && chunk == CH_)                                                      \
        return f32io ? launch_scan_t<FAM_SSD, DK_, CH_, true>(a, st)                      \
                     : launch_scan_t<FAM_SSD, DK_, CH_, false>(a, st);

hipError_t launch_scan_ssd(int dk, int chunk, bool f32io, const ScanArgs& a, hipStream_t st) {
    LKV_CASE(16, 16) LKV_CASE(32, 16) LKV_CASE(64, 16) LKV_CASE(128, 16)
    LKV_CASE(16, 64) LKV_CASE(32, 64) LKV_CASE(64, 64) LKV_CASE(128, 64)
    return hipErrorInvalidValue;
}
#undef LKV_CASE

}  // namespace lkv

// Instantiations and dispatch of the chunkwise scan kernel for the
// Gated DeltaNet family.
#include "scan_kernel.h"

namespace lkv {

#define LKV_CASE(DK_, CH_)                                                              \
    if (dk == DK_ && chunk == CH_)                                                      \
        return f32io ? launch_scan_t<FAM_GDN, DK_, CH_, true>(a, st)                      \
                     : launch_scan_t<FAM_GDN, DK_, CH_, false>(a, st);

hipError_t launch_scan_gdn(int dk, int chunk, bool f32io, const ScanArgs& a, hipStream_t st) {
    LKV_CASE(16, 16) LKV_CASE(32, 16) LKV_CASE(64, 16) LKV_CASE(128, 16)
    LKV_CASE(16, 64) LKV_CASE(32, 64) LKV_CASE(64, 64) LKV_CASE(128, 64)
    return hipErrorInvalidValue;
}
#undef LKV_CASE

}  // namespace lkv

namespace lkv {

#define LKV_LDS(FAM_, DK_, CH_)                                                            \
    if (dk == DK_ && chunk == CH_)                                                          \
        return f32io ? scan_lds_t<FAM_, DK_, CH_, true>(nw, summary)                       \
                     : scan_lds_t<FAM_, DK_, CH_, false>(nw, summary);

size_t scan_lds_bytes(int fam, int dk, int chunk, bool f32io, int nw, bool summary) {
    if (fam == FAM_GDN) {
        LKV_LDS(FAM_GDN, 16, 16) LKV_LDS(FAM_GDN, 32, 16) LKV_LDS(FAM_GDN, 64, 16) LKV_LDS(FAM_GDN, 128, 16)
        LKV_LDS(FAM_GDN, 16, 64) LKV_LDS(FAM_GDN, 32, 64) LKV_LDS(FAM_GDN, 64, 64) LKV_LDS(FAM_GDN, 128, 64)
    } else {
        LKV_LDS(FAM_SSD, 16, 16) LKV_LDS(FAM_SSD, 32, 16) LKV_LDS(FAM_SSD, 64, 16) LKV_LDS(FAM_SSD, 128, 16)
        LKV_LDS(FAM_SSD, 16, 64) LKV_LDS(FAM_SSD, 32, 64) LKV_LDS(FAM_SSD, 64, 64) LKV_LDS(FAM_SSD, 128, 64)
    }
    return 0;
}
#undef LKV_LDS

}  // namespace lkv

// Dispatch of the chunk kernel by family and mode, and its LDS footprint.
#include "chunk_kernel.h"

namespace lkv {

hipError_t launch_chunk_gdn_scan(int dk, int chunk, bool f32io, const ScanArgs& a, hipStream_t st);
hipError_t launch_chunk_gdn_summary(int dk, int chunk, bool f32io, const ScanArgs& a, hipStream_t st);
hipError_t launch_chunk_ssd_scan(int dk, int chunk, bool f32io, const ScanArgs& a, hipStream_t st);
hipError_t launch_chunk_ssd_summary(int dk, int chunk, bool f32io, const ScanArgs& a, hipStream_t st);

hipError_t launch_scan_gdn(int dk, int chunk, bool f32io, const ScanArgs& a, hipStream_t st) {
    return a.summary ? launch_chunk_gdn_summary(dk, chunk, f32io, a, st) : launch_chunk_gdn_scan(dk, chunk, f32io, a, st);
}
hipError_t launch_scan_ssd(int dk, int chunk, bool f32io, const ScanArgs& a, hipStream_t st) {
    return a.summary ? launch_chunk_ssd_summary(dk, chunk, f32io, a, st) : launch_chunk_ssd_scan(dk, chunk, f32io, a, st);
}

size_t scan_lds_bytes(int fam, int dk, int chunk, bool f32io, int nb, bool summary) {
#define LKV_LDS(FAM_, DK_, CH_)                                                              \
    if (dk == DK_ && chunk == CH_) {                                                         \
        if (!f32io) return chunk_lds_t<FAM_, DK_, CH_, false>(nb, summary);                   \
        if constexpr (DK_ <= 64) return chunk_lds_t<FAM_, DK_, CH_, true>(nb, summary);       \
        return 0;                                                                            \
    }
    if (fam == FAM_GDN) {
        LKV_LDS(FAM_GDN, 16, 16) LKV_LDS(FAM_GDN, 32, 16) LKV_LDS(FAM_GDN, 64, 16) LKV_LDS(FAM_GDN, 128, 16)
        LKV_LDS(FAM_GDN, 16, 64) LKV_LDS(FAM_GDN, 32, 64) LKV_LDS(FAM_GDN, 64, 64) LKV_LDS(FAM_GDN, 128, 64)
    } else {
        LKV_LDS(FAM_SSD, 16, 16) LKV_LDS(FAM_SSD, 32, 16) LKV_LDS(FAM_SSD, 64, 16) LKV_LDS(FAM_SSD, 128, 16)
        LKV_LDS(FAM_SSD, 16, 64) LKV_LDS(FAM_SSD, 32, 64) LKV_LDS(FAM_SSD, 64, 64) LKV_LDS(FAM_SSD, 128, 64)
    }
#undef LKV_LDS
    return 0;
}

}  // namespace lkv

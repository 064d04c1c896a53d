// Host-side launcher of the relative-error diagnostic.
#pragma once
#include "lkv_device.h"

namespace lkv {

hipError_t launch_rel_error(const float* S, const float* R, int32_t n_slices, int64_t slice_elems, int32_t group,
                            double* sq, double* rel, double* rel_group, hipStream_t st);

}  // namespace lkv

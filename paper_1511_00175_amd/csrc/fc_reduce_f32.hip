// Reduce and fused-step kernels for fp32 replicas.  The resident kernel reads
// them as pairs of 8-byte loads (FC_F32_PAIRS); the others as 16-byte loads.
#include "fc_device.h"

namespace fc {

hipError_t launch_reduce_f32(const Shape& sh, int mode, int grid, const ReduceArgs& a, hipStream_t s) {
    return launch_reduce_dt<FC_F32>(sh, mode, grid, a, s);
}

hipError_t launch_resident_f32(const Shape& sh, int mode, int grid, size_t lds, const ResidentArgs& a,
                               hipStream_t s) {
    return launch_resident_dt<FC_F32_PAIRS>(sh, mode, grid, lds, a, s);
}

hipError_t prepare_resident_f32(const Shape& sh, size_t lds) { return prepare_resident_dt<FC_F32_PAIRS>(sh, lds); }

}  // namespace fc

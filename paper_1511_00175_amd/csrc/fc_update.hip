// SGD-from-a-raw-sum and broadcast kernels: one block per tile, one thread
// per lane of the tile.
#include "fc_device.h"

namespace fc {

hipError_t launch_sgd(const Shape& sh, int grid, const SgdArgs& a, hipStream_t s) {
    auto go = [&](auto u) {
        hipLaunchKernelGGL((sgd_kernel<4, u.value>), dim3(grid), dim3(sh.lanes), 0, s, a);
        return hipGetLastError();
    };
    if (sh.vecs == 4) return go(I<4>{});
    return pick<1, 2>(sh.vecs, go);
}

hipError_t launch_bcast(const Shape& sh, int grid, const BcastArgs& a, hipStream_t s) {
    auto go = [&](auto u) {
        hipLaunchKernelGGL((bcast_kernel<4, u.value>), dim3(grid), dim3(sh.lanes), 0, s, a);
        return hipGetLastError();
    };
    if (sh.vecs == 4) return go(I<4>{});
    return pick<1, 2>(sh.vecs, go);
}

}  // namespace fc

// SGD-from-a-raw-sum and broadcast kernels: one block per tile, one thread
// per lane of the tile; on resident plans the broadcast runs one persistent
// block per CU.
#include <mutex>

#include "fc_device.h"

namespace fc {

// The raw sum between the two passes of fc_step_noalloc: a fixed array that
// the HIP runtime places on every GPU the library's code is loaded on and
// keeps until the process ends, so that the call itself allocates nothing.
// In host code `scratch` names a host-side stand-in, not device memory: its
// device address comes from hipGetSymbolAddress, once per device.
static __device__ __align__(256) float scratch[FC_NOALLOC_MAX_ELEMS];

constexpr int NOALLOC_MAX_DEVICES = 64;

hipError_t noalloc_scratch(int device, float** ptr) {
    static std::mutex mu;
    static float* address[NOALLOC_MAX_DEVICES] = {};
    if (device < 0 || device >= NOALLOC_MAX_DEVICES) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> hold(mu);
    if (!address[device]) {
        void* a = nullptr;
        const hipError_t e = hipGetSymbolAddress(&a, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!a) return hipErrorInvalidSymbol;
        address[device] = static_cast<float*>(a);
    }
    *ptr = address[device];
    return hipSuccess;
}

hipError_t launch_sgd(const Shape& sh, int grid, const SgdArgs& a, hipStream_t s) {
    auto go = [&](auto u) {
        hipLaunchKernelGGL((sgd_kernel<4, u.value>), dim3(grid), dim3(sh.block), 0, s, a);
        return hipGetLastError();
    };
    if (sh.vecs == 4) return go(I<4>{});
    return pick<1, 2>(sh.vecs, go);
}

hipError_t launch_bcast(const Shape& sh, int grid, const BcastArgs& a, hipStream_t s) {
    auto go = [&](auto u) {
        hipLaunchKernelGGL((bcast_kernel<4, u.value>), dim3(grid), dim3(sh.block), 0, s, a);
        return hipGetLastError();
    };
    if (sh.vecs == 4) return go(I<4>{});
    return pick<1, 2>(sh.vecs, go);
}

// The resident broadcast for a plan's resident tile shape (1 or 2 lane
// vectors); `lds` is the plan's LDS per block.
template <class F> hipError_t pick_resident_bcast(const Shape& sh, F&& f) {
    if (sh.block != 64) return hipErrorInvalidValue;
    if (sh.vecs == 1) return f(&resident_bcast_kernel<RESIDENT_WAVES, 1>);
    if (sh.vecs == 2) return f(&resident_bcast_kernel<RESIDENT_WAVES, 2>);
    return hipErrorInvalidValue;
}

hipError_t launch_resident_bcast(const Shape& sh, int grid, size_t lds, const BcastArgs& a, hipStream_t s) {
    return pick_resident_bcast(sh, [&](auto kernel) {
        hipLaunchKernelGGL(kernel, dim3(grid), dim3(64 * RESIDENT_WAVES), lds, s, a);
        return hipGetLastError();
    });
}

// Allow up to `lds` bytes of dynamic LDS for the kernel (a property of the
// kernel, set when a resident plan is created, like the step kernels').
hipError_t prepare_resident_bcast(const Shape& sh, size_t lds) {
    return pick_resident_bcast(sh, [&](auto kernel) {
        return hipFuncSetAttribute(reinterpret_cast<const void*>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                                   static_cast<int>(lds));
    });
}

// Read probe: a plain streaming read of one contiguous buffer, the ceiling a
// read-bound kernel can reach.  One block of 256 lanes per 16 KiB; each lane
// sums 8 pieces of 8 bytes (nt loads: measured on MI355X, the fastest plain
// read pattern found, ahead of 16-byte lanes or more bytes per lane); the
// wave and then the block add their lanes' sums and lane 0 of the block
// stores one float, which keeps the loads live.  The value's rounding order
// is not specified: it is a bandwidth probe, not a result.
constexpr int PROBE_THREADS = 256;
constexpr int PROBE_LOADS = 8;  // 8-byte loads per lane

__global__ __launch_bounds__(PROBE_THREADS) void read_probe_kernel(const void* src, uint64_t n8, float* out) {
    const uint64_t first = static_cast<uint64_t>(blockIdx.x) * PROBE_THREADS * PROBE_LOADS;
    const gptr_t base = gread(src) + first * 8;
    u2 v[PROBE_LOADS];
#pragma unroll
    for (int u = 0; u < PROBE_LOADS; ++u) {
        const uint64_t i = first + threadIdx.x + u * PROBE_THREADS;
        const uint32_t off = i < n8 ? (threadIdx.x + u * PROBE_THREADS) * 8u : 0u;
        v[u] = __builtin_bit_cast(u2, __builtin_amdgcn_raw_buffer_load_b64(rsrc((const void*)base), off, 0,
                                                                          CPOL_STREAM_LOAD));
        if (i >= n8) v[u] = u2{0u, 0u};
    }
    float x = 0.0f;
#pragma unroll
    for (int u = 0; u < PROBE_LOADS; ++u) {
        const f2 f = __builtin_bit_cast(f2, v[u]);
        x = x + (f.x + f.y);
    }
#pragma unroll
    for (int d = 32; d >= 1; d /= 2) x = x + __shfl_xor(x, d, 64);
    __shared__ float wsum[PROBE_THREADS / 64];
    if ((threadIdx.x & 63) == 0) wsum[threadIdx.x / 64] = x;
    __syncthreads();
    if (threadIdx.x == 0) {
        float t = 0.0f;
#pragma unroll
        for (int q = 0; q < PROBE_THREADS / 64; ++q) t = t + wsum[q];
        out[blockIdx.x] = t;
    }
}

uint64_t read_probe_blocks(uint64_t bytes) {
    const uint64_t per = static_cast<uint64_t>(PROBE_THREADS) * PROBE_LOADS * 8;
    return (bytes + per - 1) / per;
}

hipError_t launch_read_probe(const void* src, uint64_t bytes, float* out, hipStream_t s) {
    const uint64_t blocks = read_probe_blocks(bytes);
    hipLaunchKernelGGL(read_probe_kernel, dim3(static_cast<unsigned>(blocks)), dim3(PROBE_THREADS), 0, s, src,
                       bytes / 8, out);
    return hipGetLastError();
}

}  // namespace fc

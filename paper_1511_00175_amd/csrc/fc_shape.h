// Launch shapes and fc_step schedule chosen by default, and the (lane
// vectors, replicas per batch) pairs the kernels are compiled for.  These
// rules decide which kernel instance runs for a plan, so they live beside the
// device code.
#pragma once

#include <cstdint>

#include "fc.h"
#include "fc_internal.h"

namespace fc {

// Launch-shape defaults, measured on MI355X for the five workloads:
//   fp16 replicas       : 4 vectors per lane, 4 replicas per batch, 256 threads
//   fp32, 16 < K <= 64  : 4 vectors per lane, 2 replicas per batch, 256 threads
//   other fp32          : 1 vector per lane, 16 replicas per batch, 64 threads
// Four vectors per lane make every wave read 4 KiB of one replica at a time,
// which HBM serves better than 1 KiB pieces, as long as the lane's registers
// (16 accumulators per pending subtree) still allow enough waves in flight.
inline void default_shape(fc_dtype gdt, int K, fc::Shape& sh) {
    if (gdt == FC_F16) {
        sh.vecs = 4; sh.kchunk = 4; sh.block = 256;
    } else if (K > 16 && K <= 64) {
        sh.vecs = 4; sh.kchunk = 2; sh.block = 256;
    } else {
        sh.vecs = 1; sh.kchunk = 16; sh.block = 64;
    }
}

inline bool compiled_pair(int u, int c) {
    return (u == 1 && (c == 8 || c == 16)) || (u == 2 && (c == 8 || c == 16)) ||
           (u == 4 && (c == 2 || c == 4 || c == 8));
}

// Two passes (reduce into a raw-sum buffer, then update) when a parameter's
// replicas take more than 256 bytes: HBM serves the replica stream with one
// write stream far better than with two (measured on MI355X; see fc_schedule).
inline int default_schedule(int K, int bytes_per_element) {
    return static_cast<int64_t>(K) * bytes_per_element > 256 ? FC_SCHED_TWO_PASS : FC_SCHED_FUSED;
}

}  // namespace fc

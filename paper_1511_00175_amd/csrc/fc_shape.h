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
//   fp32, K <= 4        : 1 vector per lane, 8 replicas per batch, 256 threads
//   fp32, 16 < K <= 64  : 4 vectors per lane, 2 replicas per batch, 256 threads
//   other fp32          : 1 vector per lane, 16 replicas per batch, 64 threads
// Four vectors per lane make every wave read 4 KiB of one replica at a time,
// which HBM serves better than 1 KiB pieces, as long as the lane's registers
// (16 accumulators per pending subtree) still allow enough waves in flight.
// With at most 4 replicas a step is short and launch-bound: 4x fewer,
// larger blocks and a batch no larger than needed measured (2^20 parameters,
// us per step, steps with w, v from HBM / 20-step HIP graph on one set,
// against (1, 16, 64)): K=4 6.98-7.04 / 4.67-5.12 vs 7.58-7.79 / 4.79-5.10,
// K=2 5.78 / 4.39 vs 5.98 / 4.59; from K=8 on no better (K=8 10.68 / 7.66
// vs 10.55 / 8.09, K=16 16.47 / 14.44 vs 15.37 / 14.43).
inline void default_shape(fc_dtype gdt, int K, fc::Shape& sh) {
    if (gdt == FC_F16) {
        sh.vecs = 4; sh.kchunk = 4; sh.block = 256;
    } else if (K <= 4) {
        sh.vecs = 1; sh.kchunk = 8; sh.block = 256;
    } else if (K > 16 && K <= 64) {
        sh.vecs = 4; sh.kchunk = 2; sh.block = 256;
    } else {
        sh.vecs = 1; sh.kchunk = 16; sh.block = 64;
    }
}

// (lane vectors, replicas per batch) of the resident kernel's tiles; with
// two vectors per lane K / kchunk must stay below 128 (stack depth 7).
inline bool resident_pair(int u, int c) { return (u == 1 && c == 16) || (u == 2 && c == 4); }

// Default resident tiles: fp32 replicas with K <= 16 take 2 lane-vectors and
// batches of 4 (each wave reads 2 KiB of a replica per tile), the others 1
// lane-vector and batches of 16.  Measured on MI355X with XCD-balanced
// shares, us per step, (1, 16) vs (2, 4): VGG-19 K=16 1871-1884 vs
// 1859-1862, 40 M x K=16 534.5 vs 512.0, 40 M x K=12 427.3 vs 417.0,
// 20 M x K=8 164.1 vs 161.4, 2^20 x K=16 14.8 vs 14.1, 2^23 x K=16 98.8 vs
// 99.3; for larger K the single vector with batches of 16 keeps more bytes
// in flight per register (GoogLeNet K=128 540 vs 548, AlexNet fp16 K=128
// 2611 vs 2705, NiN K=32 equal).
inline void default_resident_shape(fc_dtype gdt, int K, int& u, int& c) {
    if (gdt == FC_F32 && K <= 16) {
        u = 2; c = 4;
    } else {
        u = 1; c = 16;
    }
}
inline bool resident_fits_k(int u, int c, int K) { return u == 1 || K / c < 128; }

// Tiles per wave whose raw sums the resident kernel keeps in registers, on
// top of the LDS slots (the plan uses them only when they save rounds: the
// kernel instance that holds them is about 4x larger).  16 waves x 4 tiles
// per CU: fp32 replicas in tiles of 2 vectors (2 KiB of sums each) with
// batches of 4 and a depth-3 pending-subtree stack (K < 32; 123 VGPRs for
// the tree step, no spill), 1.8x the parameters of LDS alone per round;
// fp16 replicas in tiles of 1 vector (1 KiB) with batches of 16 and a stack
// of depth 5 (K < 512; 92 VGPRs), 1.4x.  Measured on MI355X (us per step):
// VGG-19 K=16 in 8 rounds instead of 14, 1792 vs 1829 on one machine, 1831-1836
// vs 1861-1887 on another; AlexNet fp16 K=128 in 5 rounds instead of 6,
// 2466.9 vs 2500.2 (both builds alternated in one process; 2469 vs 2496 in
// the parameter-server order).  Not kept: 5 or 6 fp16 tiles, which give
// AlexNet 4 rounds, 2497.8 and 2511.3 vs 2469.3 and 2468.9 with 4 tiles
// (the tree step's code: 43 KB with 4 tiles, 49 KB with 5, 57 KB with 6,
// against the 64 KB instruction cache two CUs share; which limit the larger
// instances hit was not measured); 12
// unrolled tiles (106 KB of code) and rolled ones (selects that cost load
// parallelism: AlexNet fp16 in 3 rounds 2571-2576 vs 2523-2529); fp32 tiles
// of 1 vector with K < 512, 4 per wave: VGG-19-sized K=32 in 10 rounds
// instead of 14, 3098.0 vs 3117.4, 60 M x K=32 1297.5 vs 1297.7.
inline int resident_rtiles(int gdt, int u, int c, int maxd) {
    if (gdt == FC_F16 && u == 1 && c == 16 && maxd <= 5) return 4;
    return gdt == FC_F32 && u == 2 && c == 4 && maxd <= 3 ? 4 : 0;
}

inline bool compiled_pair(int u, int c) {
    return (u == 1 && (c == 8 || c == 16)) || (u == 2 && (c == 8 || c == 16)) ||
           (u == 4 && (c == 2 || c == 4 || c == 8));
}

// The resident schedule (sums parked in LDS, one persistent grid, one launch
// per round) when one round of the grid holds the whole plan, or when a
// parameter's replicas take at least 48 bytes.  Measured on MI355X (us per
// step, resident vs the best other schedule): GoogLeNet K=128 543 vs 574,
// NiN K=32 162 vs 175, VGG-19 K=16 1926 vs 1979 and K=32 3323 vs 3567 (14
// rounds), AlexNet fp16 K=32/64/128 814/1379/2574 vs 890/1535/2579 and fp32
// K=32/64 1431/2553 vs 1473/2810 (6 rounds).  With w and v kept out of the
// Infinity Cache, at 48 bytes (fp32 K=12, fp16 K=24) resident wins at every
// size tried: 143.7 M fp32 1510 vs 1634, 61 M 661 vs 673, 20 M 214 vs 227,
// 2^25 366-384 vs 374-377; fp16 61 M 675 vs 711, 2^25 373 vs 383, 20 M 217
// vs 235.  At 40 bytes the two trade places by size (within 5%), and at 32
// bytes and below the fused kernel wins or ties (fp32 K=8: 61 M 492 vs 515,
// 2^25 275 vs 293-303, 20 M 165 vs 165; fp16 K=16: 2^25 282 vs 292; VGG-19
// K=4 766 vs 846), its update writes being a larger share of the bytes.
// Steps of less than RESIDENT_MIN_BYTES of algorithmic traffic (a few
// microseconds of HBM time) stay on the single-pass fused kernel, whose one
// round trip to memory beats the resident kernel's two phases: measured on
// MI355X, us per step in a HIP graph, fused vs resident: 2^20 x K=4 (33.5 MB)
// 5.2 vs 6.6, 60000 x K=128 (31 MB) 9.5 vs 10.1, 1000 x K=1024 36.8 vs 39.1;
// from 84 MB up the resident kernel is as fast or faster (2^20 x K=16 13.0
// vs 15.0, fp16 2^20 x K=64 24.1 vs 26.4, 2^21 x K=8 15.2 vs 15.6, 200000 x
// K=256 34.4 vs 34.2).
constexpr uint64_t RESIDENT_MIN_BYTES = uint64_t(64) << 20;
inline bool default_resident(int K, int bytes_per_element, int64_t rounds, uint64_t step_bytes) {
    if (step_bytes < RESIDENT_MIN_BYTES) return false;
    return rounds == 1 || static_cast<int64_t>(K) * bytes_per_element >= 48;
}

// Resident launches record each block's rate (for fc_plan_balance) when a
// block's share of a round is at least this many tiles.  Measured on
// MI355X: the record costs about 0.6 us per launch (the timer read and the
// adds at the end of the reduce phase), 8% of a flat 2^20 x K=4 step (16
// tiles per block) and under 0.2% of the NiN-, GoogLeNet-, VGG-19- and
// AlexNet-sized steps (107-157 tiles per block), where balancing gains up to
// 1.6%.
constexpr int RESIDENT_RECORD_MIN_TILES = 32;

// Two passes (reduce into a raw-sum buffer, then update) when a parameter's
// replicas take more than 256 bytes: HBM serves the replica stream with one
// write stream far better than with two (measured on MI355X; see fc_schedule).
inline int default_schedule(int K, int bytes_per_element) {
    return static_cast<int64_t>(K) * bytes_per_element > 256 ? FC_SCHED_TWO_PASS : FC_SCHED_FUSED;
}

}  // namespace fc

// Internal interface between the host library (fc_api.cpp) and the kernels
// (fc_reduce_f32.hip, fc_reduce_f16.hip, fc_update.hip).  Not installed; the
// public ABI is include/fc.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fc {

// One block's unit of work.  A vector tile covers `count` lane-vectors of 4
// elements (count <= block_threads * vecs_per_thread) starting at element
// `start`, all inside segment `seg & SEG_MASK`.  A tail tile (bit TAIL_BIT of
// `seg` set) covers the last `count` < vector-width elements of a segment
// whose length is not a multiple of the vector width; its lanes work on one
// element each.
struct Tile {
    uint64_t start;
    uint32_t count;
    uint32_t seg;
};
static_assert(sizeof(Tile) == 16, "Tile is loaded as one 16-byte scalar load");

constexpr uint32_t TAIL_BIT = 0x80000000u;
constexpr uint32_t SEG_MASK = 0x7fffffffu;

enum Mode { MODE_REDUCE = 0, MODE_STEP = 1 };

struct Shape {
    int dtype;        // fc_dtype
    int tree;         // 1 tree order, 0 linear
    int block;        // threads per block
    int vecs;         // 4-element lane-vectors per thread (1, 2 or 4)
    int kchunk;       // replicas loaded per batch (2, 4, 8 or 16; see the pairs compiled)
    int maxd;         // depth of the pending-subtree stack (>= bit length of K / kchunk)
    int rtiles;       // resident kernel: tiles per wave whose raw sums stay in registers
};

struct ReduceArgs {
    const Tile* tiles;
    int ntiles;
    const float* mults;           // per segment j: lr_mult at 2j, decay_mult at 2j+1
    const void* const* grads;     // device table of K replica pointers
    int K;
    float* w;
    float* v;
    float* out;                   // raw sum or nullptr
    float* const* dst;            // device table of K broadcast pointers, or nullptr
    float lr, mu, wd, c;          // c = 1.0f / (float)batch
};

// The whole step in one persistent launch with the raw sums held in LDS:
// the tile map (256-element tiles: 64 lanes of one 4-element vector) is cut
// into gridDim.x * rounds contiguous ranges; in round r block b owns tiles
// [ranges[b + r * gridDim.x], ranges[b + r * gridDim.x + 1]) and reserves
// RESIDENT_SLOT floats of LDS per tile.
struct ResidentArgs {
    ReduceArgs r;
    const int* ranges;            // gridDim.x * rounds + 1 tile indices
    int rounds;
    // per block b, summed over the launches since the host last cleared it:
    // clock[4b] = tiles reduced, clock[4b + 1] = 10 ns ticks (s_memrealtime,
    // 100 MHz) of the reduce phase; clock[4b + 2] = the XCD (XCC_ID) the
    // block last ran on.  Read by the host to balance the ranges; nullptr
    // when the plan keeps equal shares (nothing is recorded).
    unsigned long long* clock;
};
constexpr int RESIDENT_CLOCK_WORDS = 4;
constexpr int RESIDENT_SLOT = 256;  // floats per tile of 64 lanes x one 4-element vector
constexpr int RESIDENT_WAVES = 16;

struct SgdArgs {
    const Tile* tiles;
    int ntiles;
    const float* mults;
    float* w;
    float* v;
    const float* g;
    float* const* dst;            // device table of K broadcast pointers, or nullptr
    int K;
    float lr, mu, wd, c;
};

struct BcastArgs {
    const Tile* tiles;
    int ntiles;
    const float* src;
    float* const* dst;
    int K;
    const int* ranges;            // resident plans: gridDim.x + 1 tile indices of one round
    int slots;                    // resident plans: LDS tile slots per block (>= 1)
};

// Largest pending-subtree stack depth compiled (stack depths 5, 7 and 10 are
// instantiated); plans whose K / kchunk needs more are rejected at creation.
constexpr int MAXD_MAX = 10;

hipError_t launch_reduce_f32(const Shape& sh, int mode, int grid, const ReduceArgs& a, hipStream_t s);
hipError_t launch_reduce_f16(const Shape& sh, int mode, int grid, const ReduceArgs& a, hipStream_t s);
hipError_t launch_sgd(const Shape& sh, int grid, const SgdArgs& a, hipStream_t s);
hipError_t launch_bcast(const Shape& sh, int grid, const BcastArgs& a, hipStream_t s);
hipError_t launch_resident_bcast(const Shape& sh, int grid, size_t lds, const BcastArgs& a, hipStream_t s);
hipError_t prepare_resident_bcast(const Shape& sh, size_t lds);
hipError_t prepare_resident_f32(const Shape& sh, size_t lds);
hipError_t prepare_resident_f16(const Shape& sh, size_t lds);
hipError_t launch_resident_f32(const Shape& sh, int mode, int grid, size_t lds, const ResidentArgs& a, hipStream_t s);
hipError_t launch_resident_f16(const Shape& sh, int mode, int grid, size_t lds, const ResidentArgs& a, hipStream_t s);
uint64_t read_probe_blocks(uint64_t bytes);

// Device address, on `device` (which must be the current device), of the
// fixed raw-sum array of fc_step_noalloc (FC_NOALLOC_MAX_ELEMS floats).
hipError_t noalloc_scratch(int device, float** ptr);
hipError_t launch_read_probe(const void* src, uint64_t bytes, float* out, hipStream_t s);

}  // namespace fc

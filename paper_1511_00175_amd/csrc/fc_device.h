// Device code of the gradient-aggregation + SGD step for gfx950 (CDNA4),
// included by the translation units that instantiate the kernels
// (fc_reduce_f32.hip, fc_reduce_f16.hip, fc_update.hip).
//
// The work is a bandwidth-bound reduction: every element of every replica is
// read once, the K values of one parameter are added in registers, and the
// parameter's weight and velocity are updated in the same pass.  Arithmetic
// intensity is at most (K + 6) flops per (4K + 16) bytes, far below the ridge
// point of the vector units, so there are no matrix-core instructions here;
// the design goals are fully coalesced loads (one 4-element vector per lane:
// 16 bytes of fp32 or 8 bytes of fp16), many loads in flight per thread, and
// a summation order that is fixed by construction.
//
// Summation order (Sec. 6.2 "Reduction tree", Fig. 3b): leaves are replicas
// 0..K-1 in order; neighbours are paired level by level and an odd last node
// moves up unchanged.  The same tree is produced by a binary counter over
// leaves: push each leaf (or each balanced subtree of kchunk consecutive
// leaves) and, while the two newest pending subtrees have equal size, replace
// them by (older + newer); at the end add the pending subtrees from the
// newest to the oldest, each older one on the left.  Pending subtrees live in
// a register stack indexed by the bit position of the counter, so every index
// is a compile-time constant after unrolling.
//
// Parameter-server order (Sec. 6.1, Fig. 3a): ((x0 + x1) + x2) + ...
//
// Update (Sec. 3, Sec. 7.1 item 2, Caffe convention):
//   ga = s*c ; d = ga + wd_j*w ; v' = mu*v + lr_j*d ; w' = w - v'
// Every operation is one rounded fp32 op: contraction is disabled below and
// the library is built with -ffp-contract=off.
//
// Kernels (all share the loads, the register stack and the epilogue, so they
// give the same bits):
//   reduce_kernel   one tile per block; reduce-only, or the fused step
//   resident_kernel one persistent block per CU: reduce a range of tiles into
//                   LDS and registers (pure reads), then finish it from there:
//                   w' stored, v' parked and stored after a barrier (or, with
//                   a broadcast, w' stored to the copies one destination at a
//                   time)
//   sgd_kernel      the update from a raw sum (second pass of two)
//   bcast_kernel    copy one vector into K destinations
//   resident_bcast_kernel  the same copy on a resident plan: a range of tiles
//                   staged in LDS, then stored one destination at a time
#pragma once

#include <type_traits>

#include "fc.h"
#include "fc_internal.h"

#pragma clang fp contract(off)

namespace fc {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef unsigned int u4 __attribute__((ext_vector_type(4)));
typedef unsigned int u2 __attribute__((ext_vector_type(2)));
typedef float f2 __attribute__((ext_vector_type(2)));
typedef _Float16 h4 __attribute__((ext_vector_type(4)));

template <int N> constexpr int ilog2() { return N <= 1 ? 0 : 1 + ilog2<N / 2>(); }

// Address spaces.  Plan tables (tiles, segment multipliers, pointer tables)
// are never written while a kernel runs: reading them through the constant
// address space lets the compiler use scalar loads.  Buffers are device
// (global) memory: replica pointers read from a table are cast to the global
// address space so that loads take the form  global_load v, v_off32, s_base.
#define FC_CONST __attribute__((address_space(4)))
#define FC_GLOBAL __attribute__((address_space(1)))

typedef const FC_GLOBAL char* gptr_t;
typedef FC_GLOBAL char* gptr_w_t;

// scalar (pointer or number) element i of a plan table
template <typename T> __device__ __forceinline__ T ldc(const T* p, int i) {
    return ((const FC_CONST T*)p)[i];
}

__device__ __forceinline__ Tile ld_tile(const Tile* tiles, int t) {
    typedef unsigned int u4_t __attribute__((ext_vector_type(4)));
    const u4_t x = ((const FC_CONST u4_t*)tiles)[t];
    Tile r;
    r.start = static_cast<uint64_t>(x.x) | (static_cast<uint64_t>(x.y) << 32);
    r.count = x.z;
    r.seg = x.w;
    return r;
}

__device__ __forceinline__ gptr_t gread(const void* p) { return (gptr_t)p; }
__device__ __forceinline__ gptr_w_t gwrite(void* p) { return (gptr_w_t)p; }

// Cache-policy bits of gfx950 buffer instructions: bit 0 = sc0, bit 1 = nt,
// bit 4 = sc1.  Replicas are read once, so their loads carry nt (streaming).
// Result stores carry sc1: measured on MI355X, this keeps the written lines
// from competing with the replica stream and is what lets two result streams
// (w' and v') ride along a 128-stream read at little cost.
constexpr int CPOL_STREAM_LOAD = 2;   // nt
constexpr int CPOL_RESULT_STORE = 16; // sc1
// The resident kernel's write phases store with their own policies: the
// update after a round's reads, which meets no read stream, with nt (measured
// on MI355X against sc1, us per step, three alternated runs each: VGG-19
// 1771-1774 vs 1790-1793, NiN 161.9-162.3 vs 163.8-164.2, GoogLeNet
// 533.6-534.0 vs 536.2-537.9); the broadcast copies with sc1 (nt: GoogLeNet
// 1180-1182 vs 1177-1180, NiN 338.4-339.4 vs 336.8-336.9).
constexpr int CPOL_RESIDENT_STORE = 2;    // nt
constexpr int CPOL_BROADCAST_STORE = 16;  // sc1

// Raw buffer resource over [base, base + 2 GiB): word 3 = 0x00020000 is the
// gfx9 data-format field for untyped 32-bit access.  Offsets used here are
// lane offsets within one tile (a few KiB).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* base) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, 0x7fffffff, 0x00020000);
}

// ------------------------------------------------------------------ replica loads
// Rep<DT, V>: V consecutive replica elements starting at element e.
template <int DT, int V> struct Rep;

// load(base, off): `base` is the replica's address of the tile's first
// element (uniform), `off` the lane's byte offset inside the tile.
template <> struct Rep<FC_F32, 4> {
    typedef f4 raw;
    __device__ static __forceinline__ raw load(gptr_t base, uint32_t off) {
        return __builtin_bit_cast(f4, __builtin_amdgcn_raw_buffer_load_b128(rsrc((const void*)base), off, 0,
                                                                           CPOL_STREAM_LOAD));
    }
    __device__ static __forceinline__ void widen(const raw& r, float* x) {
        x[0] = r.x; x[1] = r.y; x[2] = r.z; x[3] = r.w;
    }
};

template <> struct Rep<FC_F32, 1> {
    typedef float raw;
    __device__ static __forceinline__ raw load(gptr_t base, uint32_t off) {
        return *reinterpret_cast<const FC_GLOBAL float*>(base + off);
    }
    __device__ static __forceinline__ void widen(const raw& r, float* x) { x[0] = r; }
};

// fp32 replicas in the resident kernel: a lane's 4 values are two pairs of
// consecutive elements, each read with its own 8-byte load, so that each load
// instruction of a wave reads 512 contiguous bytes.  Measured on MI355X: a
// plain stream of 8-byte lane loads is 1.3-1.6% faster than one of 16-byte
// loads with the same bytes in flight, and the resident step with pairs
// 2.7% faster on NiN K=32, 0.5% on GoogLeNet K=128 and VGG-19 K=16.  The
// values stay 8-byte vectors until they are widened, so that each pair stays
// one load.  OffPair holds the two pairs' byte offsets in the tile.
constexpr int FC_F32_PAIRS = 2;
struct OffPair {
    uint32_t a, b;
};
template <> struct Rep<FC_F32_PAIRS, 4> {
    struct raw {
        u2 lo, hi;
    };
    __device__ static __forceinline__ raw load(gptr_t base, const OffPair& o) {
        raw r;
        r.lo = __builtin_bit_cast(u2, __builtin_amdgcn_raw_buffer_load_b64(rsrc((const void*)base), o.a, 0,
                                                                          CPOL_STREAM_LOAD));
        r.hi = __builtin_bit_cast(u2, __builtin_amdgcn_raw_buffer_load_b64(rsrc((const void*)base), o.b, 0,
                                                                          CPOL_STREAM_LOAD));
        return r;
    }
    __device__ static __forceinline__ void widen(const raw& r, float* x) {
        const f2 a = __builtin_bit_cast(f2, r.lo), b = __builtin_bit_cast(f2, r.hi);
        x[0] = a.x; x[1] = a.y; x[2] = b.x; x[3] = b.y;
    }
};
template <> struct Rep<FC_F32_PAIRS, 1> : Rep<FC_F32, 1> {};

// fp16 storage: binary16 -> binary32 is exact for every pattern.  A lane
// takes 4 consecutive fp16 values (8 bytes), so that the lane's fp32 weights,
// velocity and results are one 16-byte vector and every fp32 store of a wave
// covers whole cache lines.
template <> struct Rep<FC_F16, 4> {
    typedef u2 raw;
    __device__ static __forceinline__ raw load(gptr_t base, uint32_t off) {
        return __builtin_bit_cast(u2, __builtin_amdgcn_raw_buffer_load_b64(rsrc((const void*)base), off, 0,
                                                                          CPOL_STREAM_LOAD));
    }
    __device__ static __forceinline__ void widen(const raw& r, float* x) {
        const h4 h = __builtin_bit_cast(h4, r);
#pragma unroll
        for (int i = 0; i < 4; ++i) x[i] = static_cast<float>(h[i]);
    }
};

template <> struct Rep<FC_F16, 1> {
    typedef unsigned short raw;
    __device__ static __forceinline__ raw load(gptr_t base, uint32_t off) {
        return *reinterpret_cast<const FC_GLOBAL unsigned short*>(base + off);
    }
    __device__ static __forceinline__ void widen(const raw& r, float* x) {
        x[0] = static_cast<float>(__builtin_bit_cast(_Float16, r));
    }
};

// ------------------------------------------------------------------ fp32 vectors
// V fp32 results at byte offset `off`, stored with the result-store policy
template <int V, int CP = CPOL_RESULT_STORE>
__device__ __forceinline__ void st32r(gptr_w_t base, uint32_t off, const float* x) {
    if constexpr (V == 1) {
        __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned int, x[0]), rsrc((const void*)base), off, 0,
                                              CP);
    } else if constexpr (V == 2) {
        f2 t;
        t.x = x[0]; t.y = x[1];
        __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u2, t), rsrc((const void*)base), off, 0,
                                              CP);
    } else {
#pragma unroll
        for (int q = 0; q < V / 4; ++q) {
            f4 t;
            t.x = x[4 * q + 0]; t.y = x[4 * q + 1]; t.z = x[4 * q + 2]; t.w = x[4 * q + 3];
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u4, t), rsrc((const void*)base), off + 16 * q, 0,
                                                   CP);
        }
    }
}

// V fp32 values at byte offset `off`, read once (streaming policy)
template <int V> __device__ __forceinline__ void ld32s(gptr_t base, uint32_t off, float* x) {
    if constexpr (V == 1) {
        x[0] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rsrc((const void*)base), off, 0,
                                                                            CPOL_STREAM_LOAD));
    } else if constexpr (V == 2) {
        const f2 t = __builtin_bit_cast(f2, __builtin_amdgcn_raw_buffer_load_b64(rsrc((const void*)base), off, 0,
                                                                                CPOL_STREAM_LOAD));
        x[0] = t.x; x[1] = t.y;
    } else {
#pragma unroll
        for (int q = 0; q < V / 4; ++q) {
            const f4 t = __builtin_bit_cast(f4, __builtin_amdgcn_raw_buffer_load_b128(rsrc((const void*)base),
                                                                                     off + 16 * q, 0,
                                                                                     CPOL_STREAM_LOAD));
            x[4 * q + 0] = t.x; x[4 * q + 1] = t.y; x[4 * q + 2] = t.z; x[4 * q + 3] = t.w;
        }
    }
}

// ------------------------------------------------------------------ accumulators
// Partial sums are plain float[U][V] arrays, copied and added element by
// element with constant indices so that they stay in registers.
template <int U, int V> struct Acc {
    float a[U][V];
};

template <int U, int V> __device__ __forceinline__ void set(Acc<U, V>& d, const Acc<U, V>& x) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
        for (int i = 0; i < V; ++i) d.a[u][i] = x.a[u][i];
}

// d = older + d (the older, left operand first; IEEE addition is commutative,
// the order of the operands is kept only for clarity)
template <int U, int V> __device__ __forceinline__ void add_left(Acc<U, V>& d, const Acc<U, V>& older) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
        for (int i = 0; i < V; ++i) d.a[u][i] = older.a[u][i] + d.a[u][i];
}

// d = d + x
template <int U, int V> __device__ __forceinline__ void add_right(Acc<U, V>& d, const Acc<U, V>& x) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
        for (int i = 0; i < V; ++i) d.a[u][i] = d.a[u][i] + x.a[u][i];
}

// Replica k's vectors of this lane: the replica pointer comes from the plan's
// table (scalar load), the tile start is added in scalar registers.
template <int DT, int V, int U, typename O>
__device__ __forceinline__ void load_leaf(const void* const* grads, int k, uint64_t start_bytes,
                                          const O (&off)[U], typename Rep<DT, V>::raw (&r)[U]) {
    const gptr_t base = gread(ldc(grads, k)) + start_bytes;
#pragma unroll
    for (int u = 0; u < U; ++u) r[u] = Rep<DT, V>::load(base, off[u]);
}

template <int DT, int V, int U>
__device__ __forceinline__ void widen_leaf(Acc<U, V>& x, const typename Rep<DT, V>::raw (&r)[U]) {
#pragma unroll
    for (int u = 0; u < U; ++u) Rep<DT, V>::widen(r[u], x.a[u]);
}

// Binary-counter push of subtree p as subtree number `n` (0-based) onto the
// pending stack st[0..D-1]: for every bit d below the lowest clear bit t of n,
// the pending subtree st[d] (older, same size) is merged on the left; p then
// waits in st[t].  Requires n <= 2^D - 2 so that t < D.  Every branch is
// uniform and every index a constant, so the stack stays in registers.
template <int D, int U, int V>
__device__ __forceinline__ void push(Acc<U, V> (&st)[D], Acc<U, V>& p, int n) {
    const int t = __builtin_ctz(~static_cast<unsigned>(n));
#pragma unroll
    for (int d = 0; d < D; ++d) {
        if (d < t) add_left(p, st[d]);
    }
#pragma unroll
    for (int d = 0; d < D; ++d) {
        const bool here = d == t;
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int i = 0; i < V; ++i) st[d].a[u][i] = here ? p.a[u][i] : st[d].a[u][i];
    }
}

// Fold the pending subtrees named by the set bits of n into acc, newest
// (lowest bit) first, each older subtree on the left.  `have` says whether
// acc already holds a partial sum.
template <int D, int U, int V>
__device__ __forceinline__ void fold(const Acc<U, V> (&st)[D], int n, Acc<U, V>& acc, bool& have) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
        const bool take = (n >> d) & 1;
        const bool merge = take && have;
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int i = 0; i < V; ++i) {
                const float sum = st[d].a[u][i] + acc.a[u][i];
                acc.a[u][i] = merge ? sum : (take ? st[d].a[u][i] : acc.a[u][i]);
            }
        have = have || take;
    }
}

// Sum over the K replicas of V elements at e[u], u < U, in tree or linear order.
template <int DT, int V, int U, int C, int MAXD, bool TREE, typename O>
__device__ __forceinline__ void reduce(const void* const* grads, int K, uint64_t start_bytes,
                                       const O (&off)[U], Acc<U, V>& acc) {
    typedef typename Rep<DT, V>::raw raw_t;
    const int nfull = K / C;  // whole chunks of C consecutive replicas
    const int r = K - nfull * C;
    bool have = false;  // uniform across the block

    if constexpr (TREE) {
        Acc<U, V> st[MAXD];  // st[d]: pending balanced subtree of C * 2^d leaves
        for (int c = 0; c < nfull; ++c) {
            raw_t raw[C][U];
#pragma unroll
            for (int j = 0; j < C; ++j) load_leaf<DT, V, U, O>(grads, c * C + j, start_bytes, off, raw[j]);
            Acc<U, V> x[C];
#pragma unroll
            for (int j = 0; j < C; ++j) widen_leaf<DT, V, U>(x[j], raw[j]);
            // balanced subtree over the chunk, level by level: x[m] = x[2m] + x[2m+1]
#pragma unroll
            for (int h = C / 2; h >= 1; h /= 2) {
#pragma unroll
                for (int m = 0; m < h; ++m) {
                    add_right(x[2 * m], x[2 * m + 1]);
                    if (m) set(x[m], x[2 * m]);
                }
            }
            push<MAXD>(st, x[0], c);
        }
        if (r) {
            constexpr int LC = ilog2<C>();
            raw_t raw[C - 1][U];
#pragma unroll
            for (int i = 0; i < C - 1; ++i)
                if (i < r) load_leaf<DT, V, U, O>(grads, nfull * C + i, start_bytes, off, raw[i]);
            Acc<U, V> rs[LC];
#pragma unroll
            for (int i = 0; i < C - 1; ++i) {
                if (i < r) {
                    Acc<U, V> p;
                    widen_leaf<DT, V, U>(p, raw[i]);
                    push<LC>(rs, p, i);
                }
            }
            // the remainder's pending subtrees are the newest: fold them first
            fold<LC>(rs, r, acc, have);
        }
        fold<MAXD>(st, nfull, acc, have);
    } else {
        for (int c = 0; c < nfull; ++c) {
            raw_t raw[C][U];
#pragma unroll
            for (int j = 0; j < C; ++j) load_leaf<DT, V, U, O>(grads, c * C + j, start_bytes, off, raw[j]);
#pragma unroll
            for (int j = 0; j < C; ++j) {
                Acc<U, V> x;
                widen_leaf<DT, V, U>(x, raw[j]);
                if (have) add_right(acc, x);
                else set(acc, x);
                have = true;
            }
        }
        if (r) {
            raw_t raw[C - 1][U];
#pragma unroll
            for (int i = 0; i < C - 1; ++i)
                if (i < r) load_leaf<DT, V, U, O>(grads, nfull * C + i, start_bytes, off, raw[i]);
#pragma unroll
            for (int i = 0; i < C - 1; ++i) {
                if (i < r) {
                    Acc<U, V> x;
                    widen_leaf<DT, V, U>(x, raw[i]);
                    if (have) add_right(acc, x);
                    else set(acc, x);
                    have = true;
                }
            }
        }
    }
}

// One element of the momentum-SGD update; six rounded fp32 operations.
__device__ __forceinline__ void sgd1(float s, float w, float v, float lr_j, float mu, float wd_j,
                                     float c, float& wn, float& vn) {
    const float ga = s * c;
    const float decay = wd_j * w;
    const float d = ga + decay;
    const float mom = mu * v;
    const float step = lr_j * d;
    vn = mom + step;
    wn = w - vn;
}

// Lane layout inside a tile: vector u of lane t is tile vector t + u*blockDim.
// Inactive lanes point at vector 0 of the tile (always valid) and store
// nothing.  idx[u] is the lane's element index relative to the tile start.
template <int V, int U>
__device__ __forceinline__ void lane_elems(uint32_t count, uint32_t (&idx)[U], bool (&act)[U]) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const uint32_t vi = threadIdx.x + u * blockDim.x;
        act[u] = vi < count;
        idx[u] = (act[u] ? vi : 0u) * V;
    }
}

template <int DT, int V, int U, int C, int MAXD, bool TREE, int MODE>
__device__ __forceinline__ void reduce_body(const ReduceArgs& a, uint64_t start, uint32_t count,
                                            float lr_j, float wd_j) {
    constexpr uint32_t SG = DT == FC_F16 ? 2 : 4;
    uint32_t idx[U], roff[U], off[U];
    bool act[U];
    lane_elems<V, U>(count, idx, act);
#pragma unroll
    for (int u = 0; u < U; ++u) {
        roff[u] = idx[u] * SG;
        off[u] = idx[u] * 4;
    }
    const uint64_t start4 = start * 4;
    // weights and velocity are loaded before the replica stream, so that
    // their round trip to memory overlaps the replicas' (measured on MI355X:
    // a 2^20 x K=4 step in a HIP graph 4.8 vs 5.3 us, fused fp16 K=20 steps
    // 3-4% faster, fp32 K=9-10 steps equal or up to 1% faster)
    float w[U][V], v[U][V];
    if constexpr (MODE == MODE_STEP) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            ld32s<V>(gread(a.w) + start4, off[u], w[u]);
            ld32s<V>(gread(a.v) + start4, off[u], v[u]);
        }
    }
    Acc<U, V> s;
    reduce<DT, V, U, C, MAXD, TREE>(a.grads, a.K, start * SG, roff, s);
    if constexpr (MODE == MODE_REDUCE) {
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (act[u]) st32r<V>(gwrite(a.out) + start4, off[u], s.a[u]);
    } else {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (!act[u]) continue;
            float wn[V], vn[V];
#pragma unroll
            for (int i = 0; i < V; ++i) sgd1(s.a[u][i], w[u][i], v[u][i], lr_j, a.mu, wd_j, a.c, wn[i], vn[i]);
            st32r<V>(gwrite(a.w) + start4, off[u], wn);
            st32r<V>(gwrite(a.v) + start4, off[u], vn);
            if (a.out) st32r<V>(gwrite(a.out) + start4, off[u], s.a[u]);
            if (a.dst)
                for (int k = 0; k < a.K; ++k) st32r<V>(gwrite(ldc(a.dst, k)) + start4, off[u], wn);
        }
    }
}

template <int DT, int V, int U, int C, int MAXD, bool TREE, int MODE>
__global__ __launch_bounds__(256) void reduce_kernel(ReduceArgs a) {
    for (int t = blockIdx.x; t < a.ntiles; t += gridDim.x) {
        const Tile tile = ld_tile(a.tiles, t);
        float lr_j = 0.0f, wd_j = 0.0f;
        if constexpr (MODE == MODE_STEP) {
            const int j = static_cast<int>(tile.seg & SEG_MASK);
            lr_j = a.lr * ldc(a.mults, 2 * j);
            wd_j = a.wd * ldc(a.mults, 2 * j + 1);
        }
        if (!(tile.seg & TAIL_BIT))
            reduce_body<DT, V, U, C, MAXD, TREE, MODE>(a, tile.start, tile.count, lr_j, wd_j);
        else
            reduce_body<DT, 1, 1, C, MAXD, TREE, MODE>(a, tile.start, tile.count, lr_j, wd_j);
    }
}

// The end of the work on one lane-vector whose raw sum s[0..V-1] is known:
// reduce-only, store the sum; step, update w and v and store w', v' (and the
// raw sum and the broadcast copies when asked for).  KEEP (the resident
// kernel): with a broadcast, leave w' in keep[0..V-1] instead of storing the
// copies; without one, store w' and leave v' in keep[0..V-1] instead of
// storing it, for the caller to store after the block's w' stores (measured
// on MI355X with both builds alternated in one process, us per step: VGG-19
// K=16 1763.3 vs 1775.5, GoogLeNet 536.5 vs 537.7, NiN and AlexNet fp16
// unchanged).  The caller's keep may alias s.
template <int V, int MODE, bool KEEP = false, int CP = CPOL_RESULT_STORE>
__device__ __forceinline__ void finish(const ReduceArgs& a, uint64_t start4, uint32_t off, const float* s,
                                       float lr_j, float wd_j, float* keep = nullptr) {
    if constexpr (MODE == MODE_REDUCE) {
        st32r<V, CP>(gwrite(a.out) + start4, off, s);
    } else {
        float w[V], v[V], wn[V], vn[V];
        ld32s<V>(gread(a.w) + start4, off, w);
        ld32s<V>(gread(a.v) + start4, off, v);
#pragma unroll
        for (int i = 0; i < V; ++i) sgd1(s[i], w[i], v[i], lr_j, a.mu, wd_j, a.c, wn[i], vn[i]);
        st32r<V, CP>(gwrite(a.w) + start4, off, wn);
        if (!KEEP || a.dst) st32r<V, CP>(gwrite(a.v) + start4, off, vn);
        if (a.out) st32r<V, CP>(gwrite(a.out) + start4, off, s);
        if constexpr (KEEP) {
            if (a.dst) {
#pragma unroll
                for (int i = 0; i < V; ++i) keep[i] = wn[i];
            } else {
#pragma unroll
                for (int i = 0; i < V; ++i) keep[i] = vn[i];
            }
        } else if (a.dst) {
            for (int k = 0; k < a.K; ++k) st32r<V, CP>(gwrite(ldc(a.dst, k)) + start4, off, wn);
        }
    }
}

// The broadcast phase of the resident kernels: the values of the block's
// tiles [lo, hi) sit in their LDS slots (tile lo + j in slot j, parked there
// by wave j mod W), and the block stores them to the K destinations one
// destination at a time, its waves kept in step by a barrier per destination,
// so that each destination receives the block's whole range as one contiguous
// run (measured on MI355X: 3-4% faster than storing all K copies of a tile
// before the next tile).  Wave q stores the tiles whose slots it filled, so
// it reads back only what it wrote itself.  Before its slots, each wave calls
// extra(d) with the destination, to store values it holds in registers.
// Every wave of the block calls it.
template <int W, int U, class Extra>
__device__ __forceinline__ void store_slots(const Tile* tiles, float* const* dst, int K, const float* slots, int lo,
                                            int hi, Extra&& extra) {
    constexpr int SLOT = RESIDENT_SLOT * U;
    const int q = __builtin_amdgcn_readfirstlane(threadIdx.x / 64);
    const uint32_t lane = threadIdx.x & 63;
    for (int k = 0; k < K; ++k) {
        const gptr_w_t d = gwrite(ldc(dst, k));
        extra(d);
        for (int j = q; j < hi - lo; j += W) {
            const Tile tile = ld_tile(tiles, lo + j);
            const float* slot = slots + j * SLOT;
            const uint64_t start4 = tile.start * 4;
            if (!(tile.seg & TAIL_BIT)) {
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const uint32_t vi = lane + 64 * u;
                    if (vi < tile.count) st32r<4, CPOL_BROADCAST_STORE>(d + start4, vi * 16, slot + vi * 4);
                }
            } else if (lane < tile.count) {
                st32r<1, CPOL_BROADCAST_STORE>(d + start4, lane * 4, slot + lane);
            }
        }
        __syncthreads();
    }
}

// Phase 1 of the resident kernel on one tile: the raw sums of the lane's
// elements in x.  fp32 replicas (DT = FC_F32_PAIRS): the lane's values of the
// tile's elements [256 u, 256 u + 256) are the pairs at 256 u + 2 lane and
// 256 u + 128 + 2 lane (x.a[u][0..1] and x.a[u][2..3]); fp16: the lane's
// vector u is tile vector lane + 64 u.  A pair or vector past the tile's
// elements re-reads the first one.  Tail tile: the lane's element in x.a[0][0].
template <int DT, int U, int C, int MAXD, bool TREE>
__device__ __forceinline__ void reduce_tile(const ReduceArgs& a, const Tile& tile, uint32_t lane, Acc<U, 4>& x) {
    constexpr uint32_t SG = DT == FC_F16 ? 2 : 4;
    if (!(tile.seg & TAIL_BIT)) {
        if constexpr (DT == FC_F32_PAIRS) {
            const uint32_t ne = tile.count * 4;
            OffPair off[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const uint32_t e0 = 256 * u + 2 * lane, e1 = e0 + 128;
                off[u].a = (e0 < ne ? e0 : 0u) * 4;
                off[u].b = (e1 < ne ? e1 : 0u) * 4;
            }
            reduce<DT, 4, U, C, MAXD, TREE>(a.grads, a.K, tile.start * 4, off, x);
        } else {
            uint32_t off[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const uint32_t vi = lane + 64 * u;
                off[u] = (vi < tile.count ? vi : 0u) * 4 * SG;
            }
            reduce<DT, 4, U, C, MAXD, TREE>(a.grads, a.K, tile.start * SG, off, x);
        }
    } else {
        const uint32_t vi = lane < tile.count ? lane : 0u;
        const uint32_t off[1] = {vi * SG};
        Acc<1, 1> y;
        reduce<DT, 1, 1, C, MAXD, TREE>(a.grads, a.K, tile.start * SG, off, y);
        x.a[0][0] = y.a[0][0];
    }
}

// Phases 2 and 3 for a tile whose raw sums a wave kept in registers (x, in
// reduce_tile's layout: fp32 pairs, or 4-element vectors): finish the lane's
// elements (the update of w and v, or the store of the sum), leaving w' in x
// for the broadcast; and the store of w' to one destination d.
template <int DT, int U, int MODE>
__device__ __forceinline__ void finish_kept(const ReduceArgs& a, const Tile& tile, uint32_t lane, float lr_j,
                                            float wd_j, Acc<U, 4>& x) {
    const uint64_t start4 = tile.start * 4;
    if (!(tile.seg & TAIL_BIT)) {
        if constexpr (DT == FC_F32_PAIRS) {
            const uint32_t ne = tile.count * 4;  // a multiple of 4: pairs are never split
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const uint32_t e0 = 256 * u + 2 * lane, e1 = e0 + 128;
                if (e0 < ne)
                    finish<2, MODE, true, CPOL_RESIDENT_STORE>(a, start4, e0 * 4, &x.a[u][0], lr_j, wd_j, &x.a[u][0]);
                if (e1 < ne)
                    finish<2, MODE, true, CPOL_RESIDENT_STORE>(a, start4, e1 * 4, &x.a[u][2], lr_j, wd_j, &x.a[u][2]);
            }
        } else {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const uint32_t vi = lane + 64 * u;
                if (vi < tile.count)
                    finish<4, MODE, true, CPOL_RESIDENT_STORE>(a, start4, vi * 16, x.a[u], lr_j, wd_j, x.a[u]);
            }
        }
    } else if (lane < tile.count) {
        finish<1, MODE, true, CPOL_RESIDENT_STORE>(a, start4, lane * 4, &x.a[0][0], lr_j, wd_j, &x.a[0][0]);
    }
}

template <int DT, int U, int CP = CPOL_BROADCAST_STORE>
__device__ __forceinline__ void store_kept(gptr_w_t d, const Tile& tile, uint32_t lane, const Acc<U, 4>& x) {
    const uint64_t start4 = tile.start * 4;
    if (!(tile.seg & TAIL_BIT)) {
        if constexpr (DT == FC_F32_PAIRS) {
            const uint32_t ne = tile.count * 4;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const uint32_t e0 = 256 * u + 2 * lane, e1 = e0 + 128;
                if (e0 < ne) st32r<2, CP>(d + start4, e0 * 4, &x.a[u][0]);
                if (e1 < ne) st32r<2, CP>(d + start4, e1 * 4, &x.a[u][2]);
            }
        } else {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const uint32_t vi = lane + 64 * u;
                if (vi < tile.count) st32r<4, CP>(d + start4, vi * 16, x.a[u]);
            }
        }
    } else if (lane < tile.count) {
        st32r<1, CP>(d + start4, lane * 4, &x.a[0][0]);
    }
}

// ------------------------------------------------------------------ resident step
// One persistent block per CU, for each of the plan's rounds.  Phase 1: wave
// q of the block reduces tiles lo + q, lo + q + W, ... of its range in the
// same association as reduce_kernel (fp32 replicas read as 8-byte pairs,
// DT = FC_F32_PAIRS) and keeps each tile's raw sums on chip: the wave's
// first RT tiles in registers, the others in the tile's LDS slot in element
// order; HBM sees a pure read stream, no writes.  Phase 2, after a barrier:
// wave q finishes the same tiles (the SGD update, or the store of the raw
// sum), from its registers and from LDS; a step without a broadcast stores
// w' there and parks v' where the sums were, and after another barrier
// stores v' as a pure write stream; with a broadcast, phase 2 stores w' and
// v' and phase 3 stores w' to the K copies one destination at a time
// (store_slots).  The registers
// multiply what one round holds: LDS holds 160 KiB per CU, and RT tiles of
// 64 lanes x U vectors per wave add 16 * RT * U KiB.  In round r the blocks'
// ranges are neighbours, so the whole grid streams one region of the
// parameters at a time.  Blocks share nothing, so the result does not depend
// on how many of them are resident at once, nor on how the ranges divide the
// tiles.  Each block records how long its phase 1 took and on which XCD:
// blocks on some XCDs read more slowly than on others (measured on MI355X:
// 6-10%), and the host can give each block a share of tiles in proportion to
// its XCD's rate.
template <int DT, int W, int U, int C, int MAXD, bool TREE, int MODE, int RT>
__global__ __launch_bounds__(64 * W) void resident_kernel(ResidentArgs ra) {
    // 16-byte aligned, so that a lane's 4 sums move as one 16-byte LDS access
    extern __shared__ f4 slot_vecs[];
    float* slots = reinterpret_cast<float*>(slot_vecs);
    const ReduceArgs& a = ra.r;
    constexpr int SLOT = RESIDENT_SLOT * U;  // floats of LDS per tile of 64 * U vectors
    constexpr int NKEEP = RT > 0 ? RT : 1;
    const int q = __builtin_amdgcn_readfirstlane(threadIdx.x / 64);
    const uint32_t lane = threadIdx.x & 63;
    for (int round = 0; round < ra.rounds; ++round) {
        const unsigned long long t0 = ra.clock ? __builtin_amdgcn_s_memrealtime() : 0ull;
        const int b = static_cast<int>(blockIdx.x) + round * static_cast<int>(gridDim.x);
        const int lo = ldc(ra.ranges, b);
        const int hi = ldc(ra.ranges, b + 1);
        const int lo_lds = lo + W * RT;  // tile lo_lds + j sits in LDS slot j
        // phase 1: tiles lo + q + W i with i < RT into registers (the loop is
        // unrolled, so that kept[] is indexed by constants) ...
        Acc<U, 4> kept[NKEEP];
#pragma unroll
        for (int i = 0; i < RT; ++i) {
            const int t = lo + q + W * i;
            if (t < hi) reduce_tile<DT, U, C, MAXD, TREE>(a, ld_tile(a.tiles, t), lane, kept[i]);
        }
        // ... the others into LDS, in element order
        for (int t = lo_lds + q; t < hi; t += W) {
            const Tile tile = ld_tile(a.tiles, t);
            float* slot = slots + (t - lo_lds) * SLOT;
            Acc<U, 4> x;
            reduce_tile<DT, U, C, MAXD, TREE>(a, tile, lane, x);
            if (tile.seg & TAIL_BIT) {
                slot[lane] = x.a[0][0];
            } else if constexpr (DT == FC_F32_PAIRS) {
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const uint32_t e0 = 256 * u + 2 * lane, e1 = e0 + 128;
                    slot[e0] = x.a[u][0];
                    slot[e0 + 1] = x.a[u][1];
                    slot[e1] = x.a[u][2];
                    slot[e1 + 1] = x.a[u][3];
                }
            } else {
#pragma unroll
                for (int u = 0; u < U; ++u)
#pragma unroll
                    for (int i = 0; i < 4; ++i) slot[(lane + 64 * u) * 4 + i] = x.a[u][i];
            }
        }
        __syncthreads();
        if (threadIdx.x == 0 && ra.clock) {
            // how long this block's share took on its XCD (hardware register
            // XCC_ID, bits 3:0); only this block touches its entry, and the
            // adds return nothing, so the wave goes on at once
            unsigned long long* c = ra.clock + RESIDENT_CLOCK_WORDS * blockIdx.x;
            __hip_atomic_fetch_add(c, static_cast<unsigned long long>(hi - lo), __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_fetch_add(c + 1, __builtin_amdgcn_s_memrealtime() - t0, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
            c[2] = static_cast<unsigned long long>(__builtin_amdgcn_s_getreg((3 << 11) | 20));
        }
        // phase 2: the register-held tiles ...
        auto finish_reg = [&](int t, Acc<U, 4>& x) {
            const Tile tile = ld_tile(a.tiles, t);
            float lr_j = 0.0f, wd_j = 0.0f;
            if constexpr (MODE == MODE_STEP) {
                const int sj = static_cast<int>(tile.seg & SEG_MASK);
                lr_j = a.lr * ldc(a.mults, 2 * sj);
                wd_j = a.wd * ldc(a.mults, 2 * sj + 1);
            }
            finish_kept<DT, U, MODE>(a, tile, lane, lr_j, wd_j, x);  // leaves w' in x
        };
#pragma unroll
        for (int i = 0; i < RT; ++i) {
            const int t = lo + q + W * i;
            if (t < hi) finish_reg(t, kept[i]);
        }
        // ... then those in LDS, one tile per wave
        const int n = hi > lo_lds ? (hi - lo_lds) * 64 : 0;
        for (int e = static_cast<int>(threadIdx.x); e < n; e += 64 * W) {
            const int j = __builtin_amdgcn_readfirstlane(e / 64);
            const Tile tile = ld_tile(a.tiles, lo_lds + j);
            float lr_j = 0.0f, wd_j = 0.0f;
            if constexpr (MODE == MODE_STEP) {
                const int sj = static_cast<int>(tile.seg & SEG_MASK);
                lr_j = a.lr * ldc(a.mults, 2 * sj);
                wd_j = a.wd * ldc(a.mults, 2 * sj + 1);
            }
            float* slot = slots + j * SLOT;
            const uint64_t start4 = tile.start * 4;
            if (!(tile.seg & TAIL_BIT)) {
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const uint32_t vi = lane + 64 * u;
                    if (vi < tile.count)
                        finish<4, MODE, true, CPOL_RESIDENT_STORE>(a, start4, vi * 16, slot + vi * 4, lr_j, wd_j,
                                                               slot + vi * 4);
                }
            } else if (lane < tile.count) {
                finish<1, MODE, true, CPOL_RESIDENT_STORE>(a, start4, lane * 4, slot + lane, lr_j, wd_j, slot + lane);
            }
        }
        if constexpr (MODE == MODE_STEP) {
            if (!a.dst) {
                // phase 2b: v', parked in the registers and slots by phase 2,
                // stored after the block's w' stores as a pure write stream
                __syncthreads();
#pragma unroll
                for (int i = 0; i < RT; ++i) {
                    const int t = lo + q + W * i;
                    if (t < hi) store_kept<DT, U, CPOL_RESIDENT_STORE>(gwrite(a.v), ld_tile(a.tiles, t), lane, kept[i]);
                }
                for (int j = q; j < hi - lo_lds; j += W) {
                    const Tile tile = ld_tile(a.tiles, lo_lds + j);
                    const float* slot = slots + j * SLOT;
                    const uint64_t start4 = tile.start * 4;
                    if (!(tile.seg & TAIL_BIT)) {
#pragma unroll
                        for (int u = 0; u < U; ++u) {
                            const uint32_t vi = lane + 64 * u;
                            if (vi < tile.count)
                                st32r<4, CPOL_RESIDENT_STORE>(gwrite(a.v) + start4, vi * 16, slot + vi * 4);
                        }
                    } else if (lane < tile.count) {
                        st32r<1, CPOL_RESIDENT_STORE>(gwrite(a.v) + start4, lane * 4, slot + lane);
                    }
                }
            }
        }
        if constexpr (MODE == MODE_STEP) {
            // phase 3, the broadcast: w' now sits in the registers and slots
            if (a.dst)
                store_slots<W, U>(a.tiles, a.dst, a.K, slots, lo_lds, hi > lo_lds ? hi : lo_lds, [&](gptr_w_t d) {
#pragma unroll
                    for (int i = 0; i < RT; ++i) {
                        const int t = lo + q + W * i;
                        if (t < hi) store_kept<DT, U>(d, ld_tile(a.tiles, t), lane, kept[i]);
                    }
                });
        }
        __syncthreads();  // the next round's phase 1 overwrites the slots
    }
}

// ------------------------------------------------------------------ SGD from a raw sum
template <int V, int U>
__device__ __forceinline__ void sgd_body(const SgdArgs& a, uint64_t start, uint32_t count, float lr_j,
                                         float wd_j) {
    uint32_t idx[U];
    bool act[U];
    lane_elems<V, U>(count, idx, act);
    const uint64_t start4 = start * 4;
#pragma unroll
    for (int u = 0; u < U; ++u) {
        if (!act[u]) continue;
        const uint32_t off = idx[u] * 4;
        float g[V], w[V], v[V], wn[V], vn[V];
        ld32s<V>(gread(a.g) + start4, off, g);
        ld32s<V>(gread(a.w) + start4, off, w);
        ld32s<V>(gread(a.v) + start4, off, v);
#pragma unroll
        for (int i = 0; i < V; ++i) sgd1(g[i], w[i], v[i], lr_j, a.mu, wd_j, a.c, wn[i], vn[i]);
        st32r<V>(gwrite(a.w) + start4, off, wn);
        st32r<V>(gwrite(a.v) + start4, off, vn);
        if (a.dst)
            for (int k = 0; k < a.K; ++k) st32r<V>(gwrite(ldc(a.dst, k)) + start4, off, wn);
    }
}

template <int V, int U>
__global__ __launch_bounds__(256) void sgd_kernel(SgdArgs a) {
    for (int t = blockIdx.x; t < a.ntiles; t += gridDim.x) {
        const Tile tile = ld_tile(a.tiles, t);
        const int j = static_cast<int>(tile.seg & SEG_MASK);
        const float lr_j = a.lr * ldc(a.mults, 2 * j);
        const float wd_j = a.wd * ldc(a.mults, 2 * j + 1);
        if (!(tile.seg & TAIL_BIT)) sgd_body<V, U>(a, tile.start, tile.count, lr_j, wd_j);
        else sgd_body<1, 1>(a, tile.start, tile.count, lr_j, wd_j);
    }
}

// ------------------------------------------------------------------ broadcast
template <int V, int U>
__device__ __forceinline__ void bcast_body(const BcastArgs& a, uint64_t start, uint32_t count) {
    uint32_t idx[U];
    bool act[U];
    lane_elems<V, U>(count, idx, act);
    const uint64_t start4 = start * 4;
#pragma unroll
    for (int u = 0; u < U; ++u) {
        if (!act[u]) continue;
        const uint32_t off = idx[u] * 4;
        float x[V];
        ld32s<V>(gread(a.src) + start4, off, x);
        for (int k = 0; k < a.K; ++k) st32r<V>(gwrite(ldc(a.dst, k)) + start4, off, x);
    }
}

template <int V, int U>
__global__ __launch_bounds__(256) void bcast_kernel(BcastArgs a) {
    for (int t = blockIdx.x; t < a.ntiles; t += gridDim.x) {
        const Tile tile = ld_tile(a.tiles, t);
        if (!(tile.seg & TAIL_BIT)) bcast_body<V, U>(a, tile.start, tile.count);
        else bcast_body<1, 1>(a, tile.start, tile.count);
    }
}

// Broadcast on a plan with the resident schedule: one persistent block of W
// waves per CU takes its range of the round's tiles (a.ranges) in pieces of
// at most a.slots tiles (the LDS it has), its waves copy the source values of
// a piece into LDS slots (wave q the tiles lo + q, lo + q + W, ...), and the
// block stores them to the K destinations one destination at a time
// (store_slots, whose last barrier frees the slots for the next piece).
template <int W, int U>
__global__ __launch_bounds__(64 * W) void resident_bcast_kernel(BcastArgs a) {
    extern __shared__ f4 slot_vecs[];
    float* slots = reinterpret_cast<float*>(slot_vecs);
    constexpr int SLOT = RESIDENT_SLOT * U;
    const int q = __builtin_amdgcn_readfirstlane(threadIdx.x / 64);
    const uint32_t lane = threadIdx.x & 63;
    const int lo = ldc(a.ranges, blockIdx.x);
    const int hi = ldc(a.ranges, blockIdx.x + 1);
    for (int p0 = lo; p0 < hi; p0 += a.slots) {
        const int p1 = hi - p0 < a.slots ? hi : p0 + a.slots;
        for (int t = p0 + q; t < p1; t += W) {
            const Tile tile = ld_tile(a.tiles, t);
            float* slot = slots + (t - p0) * SLOT;
            const uint64_t start4 = tile.start * 4;
            if (!(tile.seg & TAIL_BIT)) {
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const uint32_t vi = lane + 64 * u;
                    if (vi < tile.count) ld32s<4>(gread(a.src) + start4, vi * 16, slot + vi * 4);
                }
            } else if (lane < tile.count) {
                ld32s<1>(gread(a.src) + start4, lane * 4, slot + lane);
            }
        }
        store_slots<W, U>(a.tiles, a.dst, a.K, slots, p0, p1, [](gptr_w_t) {});
    }
}

// ------------------------------------------------------------------ dispatch
template <int N> using I = std::integral_constant<int, N>;

template <int A, int B, class F> hipError_t pick(int x, F&& f) {
    return x == B ? f(I<B>{}) : f(I<A>{});
}

// Pending-subtree stack depths compiled (>= bit length of K / kchunk).
template <class F> hipError_t pick_maxd(int maxd, F&& f) {
    if (maxd <= 5) return f(I<5>{});
    if (maxd <= 7) return f(I<7>{});
    return f(I<MAXD_MAX>{});
}

// (vectors per lane, replicas per batch) pairs compiled.
template <class F> hipError_t pick_uc(int u, int c, F&& f) {
    if (u == 1 && c == 16) return f(I<1>{}, I<16>{});
    if (u == 1 && c == 8) return f(I<1>{}, I<8>{});
    if (u == 2 && c == 16) return f(I<2>{}, I<16>{});
    if (u == 2 && c == 8) return f(I<2>{}, I<8>{});
    if (u == 4 && c == 8) return f(I<4>{}, I<8>{});
    if (u == 4 && c == 4) return f(I<4>{}, I<4>{});
    if (u == 4 && c == 2) return f(I<4>{}, I<2>{});
    return hipErrorInvalidValue;
}

template <int DT, int TREE, int MODE, int U, int C, int MAXD>
hipError_t go_reduce(int grid, int block, const ReduceArgs& a, hipStream_t s) {
    constexpr int V = 4;  // elements per lane-vector for both storage types
    hipLaunchKernelGGL((reduce_kernel<DT, V, U, C, MAXD, (TREE != 0), MODE>), dim3(grid), dim3(block), 0, s, a);
    return hipGetLastError();
}

template <int DT>
hipError_t launch_reduce_dt(const Shape& sh, int mode, int grid, const ReduceArgs& a, hipStream_t s) {
    return pick<MODE_REDUCE, MODE_STEP>(mode, [&](auto md) {
        return pick_uc(sh.vecs, sh.kchunk, [&](auto u, auto c) {
            if (sh.tree) {
                return pick_maxd(sh.maxd, [&](auto d) {
                    return go_reduce<DT, 1, md.value, u.value, c.value, d.value>(grid, sh.block, a, s);
                });
            }
            return go_reduce<DT, 0, md.value, u.value, c.value, 1>(grid, sh.block, a, s);
        });
    });
}

// The resident kernel instance for a plan's shape: f(kernel instance tag).
// The register-held tiles per wave (sh.rtiles) are the plan's
// (resident_rtiles): its rounds are sized for them.
template <int DT, class F> hipError_t pick_resident(const Shape& sh, int mode, F&& f) {
    if (sh.block != 64) return hipErrorInvalidValue;
    auto go = [&](auto u, auto c, auto d, auto rt) {
        return pick<MODE_REDUCE, MODE_STEP>(mode, [&](auto md) {
            if (sh.tree)
                return f(&resident_kernel<DT, RESIDENT_WAVES, u.value, c.value, d.value, true, md.value, rt.value>);
            return f(&resident_kernel<DT, RESIDENT_WAVES, u.value, c.value, d.value, false, md.value, rt.value>);
        });
    };
    constexpr bool pairs = DT == FC_F32_PAIRS;
    // (lane vectors, replicas per batch) of the resident tiles; two vectors
    // per lane only with stacks up to depth 7 (deeper ones would spill)
    if (sh.vecs == 1 && sh.kchunk == 16) {
        if constexpr (DT == FC_F16) {
            if (sh.rtiles == 4 && sh.maxd <= 5) return go(I<1>{}, I<16>{}, I<5>{}, I<4>{});
        }
        if (sh.rtiles != 0) return hipErrorInvalidValue;
        return pick_maxd(sh.maxd, [&](auto d) { return go(I<1>{}, I<16>{}, d, I<0>{}); });
    }
    if (sh.vecs == 2 && sh.kchunk == 4) {
        if constexpr (pairs) {
            if (sh.rtiles == 4 && sh.maxd <= 3) return go(I<2>{}, I<4>{}, I<3>{}, I<4>{});
        }
        if (sh.rtiles != 0) return hipErrorInvalidValue;
        if (sh.maxd <= 5) return go(I<2>{}, I<4>{}, I<5>{}, I<0>{});
        if (sh.maxd <= 7) return go(I<2>{}, I<4>{}, I<7>{}, I<0>{});
    }
    return hipErrorInvalidValue;
}

// Allow up to `lds` bytes of dynamic LDS for the plan's resident kernels
// (both modes) on the current device; called when a plan is created.  The
// limit is a property of the kernel, shared by every plan that uses it.
template <int DT>
hipError_t prepare_resident_dt(const Shape& sh, size_t lds) {
    for (int mode : {static_cast<int>(MODE_REDUCE), static_cast<int>(MODE_STEP)}) {
        const hipError_t e = pick_resident<DT>(sh, mode, [&](auto kernel) {
            return hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
        });
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

template <int DT>
hipError_t launch_resident_dt(const Shape& sh, int mode, int grid, size_t lds, const ResidentArgs& a,
                              hipStream_t s) {
    return pick_resident<DT>(sh, mode, [&](auto kernel) {
        hipLaunchKernelGGL(kernel, dim3(grid), dim3(64 * RESIDENT_WAVES), lds, s, a);
        return hipGetLastError();
    });
}

}  // namespace
}  // namespace fc

// Host side of the C ABI declared in include/fc.h: plan construction (tile
// map, segment multipliers, replica pointer tables), argument validation and
// kernel launch.  Every call validates before it enqueues anything.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <new>
#include <vector>

#include "fc.h"
#include "fc_internal.h"
#include "fc_partition.h"
#include "fc_shape.h"

using fc::Tile;

struct fc_plan {
    int K = 0;
    fc_dtype gdt = FC_F32;
    fc_order order = FC_ORDER_TREE;
    int vec = 4;        // elements per lane-vector (16 bytes of fp32, 8 bytes of fp16)
    int sg = 4;         // bytes per replica element
    std::vector<fc_segment> segs;
    uint64_t n_elems = 0;
    uint64_t extent = 0;  // one past the last segment element
    fc::Shape shape{};
    int ntiles = 0;
    int grid = 0;
    int device = 0;

    Tile* d_tiles = nullptr;
    float* d_mults = nullptr;
    const void** d_grads = nullptr;  // K replica pointers
    float** d_dst = nullptr;         // K broadcast pointers
    float* d_sum = nullptr;          // raw-sum scratch of the two-pass schedule (extent floats)
    int schedule = FC_SCHED_FUSED;   // resolved schedule of fc_step
    int* d_ranges = nullptr;         // RESIDENT: tile range of each block in each round (res_grid * res_rounds + 1)
    int res_grid = 0;
    int res_rounds = 0;
    bool res_one_launch = false;     // every round in one launch (FC_SCHED_RESIDENT_ONE_LAUNCH)
    int res_lds = 0;                 // RESIDENT: LDS bytes per block
    int res_slot = 0;                // RESIDENT: LDS bytes per tile
    int res_in_regs = 0;             // RESIDENT: tiles per block held in registers
    bool res_record = false;         // RESIDENT: launches record per-block rates into d_clock
    std::vector<int> res_ranges;     // RESIDENT: host copy of the d_ranges table
    unsigned long long* d_clock = nullptr;  // RESIDENT: per block, the kernel's phase-1 clock and XCD


    // per-kernel timing (fc_plan_set_timing / fc_plan_read_timing)
    struct Rec {
        hipEvent_t a, b;
        int kind;
    };
    bool timing = false;
    std::vector<hipEvent_t> event_pool;
    std::vector<Rec> records;

    // host copies of what the device pointer tables hold (valid flags)
    std::vector<const void*> h_grads;
    std::vector<float*> h_dst;
    bool grads_valid = false;
    bool dst_valid = false;
    hipStream_t last_stream = nullptr;  // stream of the plan's previous (uncaptured) call
    bool have_last_stream = false;
    hipEvent_t order_event = nullptr;    // orders a call on another stream after the previous one
                                         // (created with the plan: no call creates anything)
};

namespace {

constexpr int K_MAX = 1024;

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

struct Span {
    uintptr_t lo, hi;  // [lo, hi)
    int id;            // distinct buffer id; replicas share role 0 and differ by id
    bool written;
    bool replica;
};

// The buffers one call names (at most K replicas, K destinations and four
// more), held on the caller's stack so that validation allocates nothing.
struct Spans {
    static constexpr int CAP = 2 * K_MAX + 4;
    Span v[CAP];
    int n = 0;
    void push(const Span& x) { v[n++] = x; }
};

// Written buffers may not overlap any other buffer, except that `out` may be
// exactly a replica of an FC_F32 plan (each element is read by the thread
// that writes it).  Read-only buffers may overlap each other.  The spans are
// sorted by start and each is compared only with the spans that start
// before it ends, so a valid call costs O(n log n) for n = K + a few spans.
int check_aliasing(Spans& sp, int out_id, bool f32) {
    Span* spans = sp.v;
    const size_t n =
        static_cast<size_t>(std::remove_if(spans, spans + sp.n, [](const Span& x) { return x.hi == x.lo; }) - spans);
    std::sort(spans, spans + n, [](const Span& x, const Span& y) { return x.lo < y.lo; });
    for (size_t i = 0; i < n; ++i) {
        const Span& a = spans[i];
        for (size_t j = i + 1; j < n && spans[j].lo < a.hi; ++j) {
            const Span& b = spans[j];  // overlaps a: b.lo >= a.lo and b.lo < a.hi
            if (!a.written && !b.written) continue;
            const bool exact_out_alias =
                f32 && ((a.id == out_id && b.replica) || (b.id == out_id && a.replica)) && a.lo == b.lo &&
                a.hi == b.hi;
            if (!exact_out_alias) return FC_EALIAS;
        }
    }
    return FC_OK;
}

int hip_rc(hipError_t e) { return e == hipSuccess ? FC_OK : FC_EHIP; }

// FC_OK when `s` is not being captured into a graph; FC_EINVAL when it is
// (a host wait on it, a table copy or a timed launch would break or corrupt
// the capture).
int capture_check(hipStream_t s) {
    hipStreamCaptureStatus st = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(s, &st) != hipSuccess) return FC_EHIP;
    return st == hipStreamCaptureStatusNone ? FC_OK : FC_EINVAL;
}

// Calls on one plan take effect in the order they are made, whatever their
// streams.  A call on another stream than the plan's previous call first
// makes its stream wait, on the device, for everything enqueued so far on
// the previous call's stream (one event recorded there), so the plan's
// shared device state -- pointer tables, the two-pass raw-sum scratch, the
// resident launch record -- never serves two calls at once and the host
// never waits.  A call enqueued while its stream is being captured into a
// graph runs when the graph is launched, which its launcher orders: it
// neither waits nor becomes the previous call.  Sets `note` when the call
// becomes the plan's previous call (note_stream once it has enqueued).
int order_after_last(fc_plan* p, hipStream_t s, bool& note) {
    note = false;
    if (p->have_last_stream && p->last_stream == s) return FC_OK;
    int rc = capture_check(s);
    if (rc == FC_EINVAL) return FC_OK;  // being captured
    if (rc) return rc;
    note = true;
    if (!p->have_last_stream) return FC_OK;
    // the previous stream's pending work cannot be named by an event recorded
    // outside a capture it has since joined
    rc = capture_check(p->last_stream);
    if (rc) return rc;
    if (hipEventRecord(p->order_event, p->last_stream) != hipSuccess ||
        hipStreamWaitEvent(s, p->order_event, 0) != hipSuccess)
        return FC_EHIP;
    return FC_OK;
}

// Replace a device pointer table if its contents differ from the last call.
// The copy is ordered on `s` after every earlier call of the plan
// (order_after_last ran first).  Not while `s` is being captured into a
// graph: the graph would record a copy from the plan's host buffer, which
// later calls overwrite, so a capture may only hold calls that keep the
// tables.  `host` has K entries from plan creation on, so assigning K new
// ones allocates nothing.
template <typename P>
int update_table(fc_plan* p, std::vector<P>& host, bool& valid, P* dev, const P* want, hipStream_t s) {
    const size_t K = static_cast<size_t>(p->K);
    if (valid && std::equal(host.begin(), host.end(), want)) return FC_OK;
    const int rc = capture_check(s);
    if (rc) return rc;
    host.assign(want, want + K);
    valid = false;
    if (hipMemcpyAsync(dev, host.data(), K * sizeof(P), hipMemcpyHostToDevice, s) != hipSuccess)
        return FC_EHIP;
    valid = true;
    return FC_OK;
}

hipError_t launch_reduce(const fc::Shape& sh, int mode, int grid, const fc::ReduceArgs& a, hipStream_t s) {
    return sh.dtype == FC_F16 ? fc::launch_reduce_f16(sh, mode, grid, a, s) : fc::launch_reduce_f32(sh, mode, grid, a, s);
}

// One launch per round: the kernel boundary keeps the whole grid in step, so
// one round's update writes never meet the next round's replica reads
// (measured on MI355X, VGG-19 K=16 in 14 rounds: 1881 us vs 2076 us with
// all rounds in one launch).  A plan made for one launch gives the kernel
// every round: block b then takes range b + grid * round in turn.
hipError_t launch_resident(fc_plan* p, int mode, const fc::ReduceArgs& r, hipStream_t s) {
    fc::ResidentArgs a{};
    a.r = r;
    a.rounds = p->res_one_launch ? p->res_rounds : 1;
    a.clock = p->res_record ? p->d_clock : nullptr;
    const size_t lds = static_cast<size_t>(p->res_lds);
    for (int round = 0; round < p->res_rounds; round += a.rounds) {
        a.ranges = p->d_ranges + static_cast<size_t>(round) * p->res_grid;
        const hipError_t e = p->shape.dtype == FC_F16
                                 ? fc::launch_resident_f16(p->shape, mode, p->res_grid, lds, a, s)
                                 : fc::launch_resident_f32(p->shape, mode, p->res_grid, lds, a, s);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

// Zero the per-block record of the resident launches (synchronous).
hipError_t clear_clock(fc_plan* p) {
    try {
        std::vector<unsigned long long> z(static_cast<size_t>(p->res_grid) * fc::RESIDENT_CLOCK_WORDS, 0ull);
        return hipMemcpy(p->d_clock, z.data(), z.size() * sizeof(unsigned long long), hipMemcpyHostToDevice);
    } catch (const std::bad_alloc&) {
        return hipErrorOutOfMemory;  // no exception leaves the C ABI
    }
}

void note_stream(fc_plan* p, hipStream_t s) {
    p->last_stream = s;
    p->have_last_stream = true;
}

int validate_opts(const fc_launch_opts* o, fc_dtype gdt, int K, fc::Shape& sh, bool& shape_given) {
    fc::default_shape(gdt, K, sh);
    shape_given = false;
    if (o) {
        // k_waves: one wave reduces all K replicas of its lane-vectors (0 or 1)
        if (o->k_waves < 0 || o->k_waves > 1 || o->max_blocks < 0) return FC_EINVAL;
        if (o->schedule < FC_SCHED_AUTO || o->schedule > FC_SCHED_RESIDENT_ONE_LAUNCH) return FC_EINVAL;
        shape_given = o->block_threads || o->vecs_per_thread || o->kchunk || o->k_waves;
        if (o->schedule == FC_SCHED_RESIDENT || o->schedule == FC_SCHED_RESIDENT_ONE_LAUNCH) {
            // the resident kernel's tiles: 64 lanes of (1 vector, batches of 16)
            // or (2 vectors, batches of 4).  The plan sets the shape.
            const int ru = o->vecs_per_thread ? o->vecs_per_thread : 1;
            const int rc = o->kchunk ? o->kchunk : (ru == 2 ? 4 : 16);
            if ((o->block_threads && o->block_threads != 64) || !fc::resident_pair(ru, rc) ||
                !fc::resident_fits_k(ru, rc, K))
                return FC_EINVAL;
            return FC_OK;
        }
        if (o->block_threads) {
            if (o->block_threads != 64 && o->block_threads != 128 && o->block_threads != 256) return FC_EINVAL;
            sh.block = o->block_threads;
        }
        if (o->vecs_per_thread || o->kchunk) {
            // an explicit pair replaces the default pair; one field alone keeps the other default
            const int pu = o->vecs_per_thread ? o->vecs_per_thread : sh.vecs;
            const int pc = o->kchunk ? o->kchunk : sh.kchunk;
            if (!fc::compiled_pair(pu, pc)) return FC_EINVAL;
            sh.vecs = pu;
            sh.kchunk = pc;
        }
    }
    return FC_OK;
}

int bit_length(int x) {
    int n = 0;
    while (x > 0) {
        ++n;
        x >>= 1;
    }
    return n;
}

void free_plan(fc_plan* p) {
    if (!p) return;
    for (auto& r : p->records) {
        (void)hipEventDestroy(r.a);
        (void)hipEventDestroy(r.b);
    }
    for (auto e : p->event_pool) (void)hipEventDestroy(e);
    if (p->order_event) (void)hipEventDestroy(p->order_event);
    if (p->d_sum) (void)hipFree(p->d_sum);
    if (p->d_ranges) (void)hipFree(p->d_ranges);
    if (p->d_clock) (void)hipFree(p->d_clock);
    if (p->d_tiles) (void)hipFree(p->d_tiles);
    if (p->d_mults) (void)hipFree(p->d_mults);
    if (p->d_grads) (void)hipFree(p->d_grads);
    if (p->d_dst) (void)hipFree(p->d_dst);
    delete p;
}

hipError_t take_event(fc_plan* p, hipEvent_t* e) {
    if (!p->event_pool.empty()) {
        *e = p->event_pool.back();
        p->event_pool.pop_back();
        return hipSuccess;
    }
    return hipEventCreate(e);
}

// Launch `go` on stream s; with timing on, bracket it with two events (not
// while s is being captured: the plan's records would then name events that
// only a graph records, so such a call is refused before anything is enqueued).
template <typename F>
int launch(fc_plan* p, int kind, hipStream_t s, F&& go) {
    if (!p->timing) return hip_rc(go());
    const int crc = capture_check(s);
    if (crc) return crc;
    fc_plan::Rec r{nullptr, nullptr, kind};
    if (take_event(p, &r.a) != hipSuccess) return FC_EHIP;
    if (take_event(p, &r.b) != hipSuccess) {
        p->event_pool.push_back(r.a);
        return FC_EHIP;
    }
    try {
        p->records.reserve(p->records.size() + 1);
    } catch (const std::bad_alloc&) {
        p->event_pool.push_back(r.a);
        p->event_pool.push_back(r.b);
        return FC_ENOMEM;
    }
    if (hipEventRecord(r.a, s) != hipSuccess) {
        p->event_pool.push_back(r.a);
        p->event_pool.push_back(r.b);
        return FC_EHIP;
    }
    const int rc = hip_rc(go());
    if (hipEventRecord(r.b, s) != hipSuccess) {
        // the start event may still complete; both go back to the pool unused
        p->event_pool.push_back(r.a);
        p->event_pool.push_back(r.b);
        return FC_EHIP;
    }
    p->records.push_back(r);
    return rc;
}

// Every entry point returns a code: a host allocation that fails inside one
// (validation spans, pointer-table copies, event bookkeeping) is FC_ENOMEM,
// and no exception leaves the C ABI.
template <typename F>
int guarded(F&& body) {
    try {
        return body();
    } catch (const std::bad_alloc&) {
        return FC_ENOMEM;
    } catch (...) {
        return FC_EHIP;
    }
}

}  // namespace

extern "C" {

const char* fc_strerror(int code) {
    switch (code) {
        case FC_OK: return "success";
        case FC_EINVAL: return "invalid argument";
        case FC_EALIGN: return "misaligned pointer or segment offset";
        case FC_EALIAS: return "a written buffer overlaps another buffer";
        case FC_EHIP: return "HIP runtime error";
        case FC_ENOMEM: return "out of host memory";
        case FC_ESIZE: return "plan larger than the fixed raw-sum array of fc_step_noalloc";
        default: return "unknown error code";
    }
}

int fc_plan_create_ex(fc_plan** plan, const fc_segment* segs, int nseg, int K, int gdt_in, int order_in,
                      const fc_launch_opts* opts) {
    if (!plan) return FC_EINVAL;
    *plan = nullptr;
    if (nseg < 0 || (nseg > 0 && !segs)) return FC_EINVAL;
    if (K < 1 || K > K_MAX) return FC_EINVAL;
    if (gdt_in != FC_F32 && gdt_in != FC_F16) return FC_EINVAL;
    if (order_in != FC_ORDER_TREE && order_in != FC_ORDER_LINEAR) return FC_EINVAL;
    const fc_dtype gdt = static_cast<fc_dtype>(gdt_in);
    const fc_order order = static_cast<fc_order>(order_in);
    const int vec = 4;
    uint64_t end = 0, n_elems = 0;
    for (int j = 0; j < nseg; ++j) {
        const fc_segment& s = segs[j];
        if (s.offset % static_cast<uint64_t>(vec)) return FC_EALIGN;
        if (s.length > UINT64_MAX - s.offset) return FC_EINVAL;
        if (j > 0 && s.offset < end) return FC_EINVAL;  // unsorted or overlapping
        end = std::max(end, s.offset + s.length);
        n_elems += s.length;
    }
    // byte offsets of every element must fit in 64 bits for every buffer
    if (end > (UINT64_MAX / 8)) return FC_EINVAL;
    fc::Shape sh{};
    bool shape_given = false;
    int rc = validate_opts(opts, gdt, K, sh, shape_given);
    if (rc) return rc;
    const int sched_req = opts ? opts->schedule : FC_SCHED_AUTO;
    const bool res_req = sched_req == FC_SCHED_RESIDENT || sched_req == FC_SCHED_RESIDENT_ONE_LAUNCH;

    // RESIDENT: one block per compute unit; each round every block takes a
    // range of 256-element tiles whose raw sums fit the compute unit's LDS
    int device = 0, cus = 0, lds_cu = 0;
    if (hipGetDevice(&device) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess ||
        hipDeviceGetAttribute(&lds_cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, device) != hipSuccess)
        return FC_EHIP;
    int res_u = 1, res_c = 16;  // the resident tiles' lane vectors and batch
    fc::default_resident_shape(gdt, K, res_u, res_c);
    if (res_req && opts->vecs_per_thread) {
        res_u = opts->vecs_per_thread;
        res_c = opts->kchunk ? opts->kchunk : (res_u == 2 ? 4 : 16);
    } else if (res_req && opts->kchunk) {
        // a batch alone names single-vector tiles, as validate_opts checks
        res_u = 1;
        res_c = opts->kchunk;
    }
    const uint64_t tile_vecs_r = 64 * static_cast<uint64_t>(res_u);
    uint64_t res_tiles = 0;
    for (int j = 0; j < nseg; ++j)
        res_tiles += (segs[j].length / vec + tile_vecs_r - 1) / tile_vecs_r + (segs[j].length % vec ? 1 : 0);
    const uint64_t slot_bytes = fc::RESIDENT_SLOT * sizeof(float) * res_u;
    const uint64_t cap_lds = std::max<uint64_t>(1, static_cast<uint64_t>(std::max(lds_cu, 0)) / slot_bytes);
    int res_grid = std::max(1, cus);
    if (opts && opts->max_blocks > 0) res_grid = std::min(res_grid, opts->max_blocks);
    if (res_tiles > 0 && res_tiles < static_cast<uint64_t>(res_grid)) res_grid = static_cast<int>(res_tiles);
    auto rounds_for = [&](uint64_t per_block) {
        const uint64_t per_round = static_cast<uint64_t>(res_grid) * per_block;
        return std::max<uint64_t>(1, (res_tiles + per_round - 1) / per_round);
    };
    // a block's tiles in one round: the waves' register-held tiles first,
    // then LDS slots; the register-held tiles are used only when they save
    // rounds (their kernel instance is larger)
    int res_rt = fc::resident_rtiles(gdt, res_u, res_c, bit_length(K / res_c));
    if (res_rt > 0 && rounds_for(cap_lds + static_cast<uint64_t>(fc::RESIDENT_WAVES) * res_rt) >= rounds_for(cap_lds))
        res_rt = 0;
    const uint64_t in_regs = static_cast<uint64_t>(fc::RESIDENT_WAVES) * res_rt;
    const uint64_t cap = cap_lds + in_regs;
    const uint64_t res_rounds = rounds_for(cap);
    const uint64_t res_ranges = static_cast<uint64_t>(res_grid) * res_rounds;
    // LDS for the most tiles a block may ever hold beyond its registers, so
    // that rebalanced ranges (fc_plan_balance) never need more than a launch
    // already has, also in a captured graph (measured on MI355X: the size
    // itself does not change the speed)
    const uint64_t most = std::min<uint64_t>(cap, std::max<uint64_t>(1, (res_tiles + res_rounds - 1) / res_rounds));
    const uint64_t res_lds = std::max<uint64_t>(1, most > in_regs ? most - in_regs : 0) * slot_bytes;
    if (res_ranges > static_cast<uint64_t>(INT32_MAX) - 1) return FC_EINVAL;
    // algorithmic bytes of one step (saturating)
    const uint64_t per_elem = static_cast<uint64_t>(K) * (gdt == FC_F16 ? 2 : 4) + 16;
    const uint64_t step_bytes = n_elems > UINT64_MAX / per_elem ? UINT64_MAX : n_elems * per_elem;
    const bool resident =
        res_req ||
        (sched_req == FC_SCHED_AUTO && !shape_given &&
         fc::default_resident(K, gdt == FC_F16 ? 2 : 4, static_cast<int64_t>(res_rounds), step_bytes));
    if (resident) {
        sh.block = 64;
        sh.vecs = res_u;
        sh.kchunk = res_c;
        sh.rtiles = res_rt;
    }

    fc_plan* p = new (std::nothrow) fc_plan();
    if (!p) return FC_ENOMEM;
    p->K = K;
    p->gdt = gdt;
    p->order = order;
    p->vec = vec;
    p->sg = gdt == FC_F16 ? 2 : 4;
    p->n_elems = n_elems;
    p->extent = end;
    sh.dtype = gdt;
    sh.tree = order == FC_ORDER_TREE;
    sh.maxd = bit_length(K / sh.kchunk);
    if (sh.maxd > fc::MAXD_MAX) {
        delete p;
        return FC_EINVAL;
    }
    p->shape = sh;

    // Tile map: each segment is cut into tiles of at most block*vecs vectors;
    // a length that is not a multiple of the vector width leaves a tail tile.
    std::vector<Tile> tiles;
    std::vector<float> mults;
    try {
        p->segs.assign(segs, segs + nseg);
        mults.resize(2 * static_cast<size_t>(std::max(nseg, 1)));
        const uint64_t tile_vecs = static_cast<uint64_t>(sh.block) * sh.vecs;
        for (int j = 0; j < nseg; ++j) {
            const fc_segment& s = segs[j];
            mults[2 * j] = s.lr_mult;
            mults[2 * j + 1] = s.decay_mult;
            const uint64_t nvec = s.length / vec;
            const uint64_t tail = s.length % vec;
            for (uint64_t v0 = 0; v0 < nvec; v0 += tile_vecs) {
                Tile t;
                t.start = s.offset + v0 * vec;
                t.count = static_cast<uint32_t>(std::min(tile_vecs, nvec - v0));
                t.seg = static_cast<uint32_t>(j);
                tiles.push_back(t);
            }
            if (tail) {
                Tile t;
                t.start = s.offset + nvec * vec;
                t.count = static_cast<uint32_t>(tail);
                t.seg = static_cast<uint32_t>(j) | fc::TAIL_BIT;
                tiles.push_back(t);
            }
        }
        p->h_grads.assign(K, nullptr);
        p->h_dst.assign(K, nullptr);
    } catch (const std::bad_alloc&) {
        delete p;
        return FC_ENOMEM;
    }
    if (tiles.size() > static_cast<size_t>(INT32_MAX)) {
        delete p;
        return FC_EINVAL;
    }
    p->ntiles = static_cast<int>(tiles.size());
    int grid = p->ntiles;
    if (opts && opts->max_blocks > 0) grid = std::min(grid, opts->max_blocks);
    p->grid = grid;

    // fc_step schedule (see fc_schedule)
    if (resident) p->schedule = FC_SCHED_RESIDENT;
    else p->schedule = sched_req == FC_SCHED_AUTO ? fc::default_schedule(K, p->sg) : sched_req;
    p->device = device;
    std::vector<int>& ranges = p->res_ranges;
    if (resident) {
        p->res_grid = res_grid;
        p->res_rounds = static_cast<int>(res_rounds);
        p->res_one_launch = sched_req == FC_SCHED_RESIDENT_ONE_LAUNCH;
        p->res_lds = static_cast<int>(res_lds);
        p->res_slot = static_cast<int>(slot_bytes);
        p->res_in_regs = static_cast<int>(in_regs);
        p->res_record = (res_tiles + res_ranges - 1) / res_ranges >= static_cast<uint64_t>(fc::RESIDENT_RECORD_MIN_TILES);
        try {
            ranges.resize(static_cast<size_t>(res_ranges) + 1);
        } catch (const std::bad_alloc&) {
            delete p;
            return FC_ENOMEM;
        }
        fc::equal_ranges(p->ntiles, p->res_rounds, res_grid, ranges);
    }

    bool ok = hipEventCreateWithFlags(&p->order_event, hipEventDisableTiming) == hipSuccess &&
              hipMalloc(&p->d_tiles, std::max<size_t>(tiles.size(), 1) * sizeof(Tile)) == hipSuccess &&
              hipMalloc(&p->d_mults, mults.size() * sizeof(float)) == hipSuccess &&
              hipMalloc(reinterpret_cast<void**>(&p->d_grads), K * sizeof(void*)) == hipSuccess &&
              hipMalloc(reinterpret_cast<void**>(&p->d_dst), K * sizeof(float*)) == hipSuccess;
    if (ok && p->schedule == FC_SCHED_TWO_PASS && p->extent > 0)
        ok = hipMalloc(&p->d_sum, static_cast<size_t>(p->extent) * sizeof(float)) == hipSuccess;
    if (ok && resident) {
        const size_t clock_bytes = static_cast<size_t>(res_grid) * fc::RESIDENT_CLOCK_WORDS * sizeof(unsigned long long);
        ok = hipMalloc(reinterpret_cast<void**>(&p->d_ranges), ranges.size() * sizeof(int)) == hipSuccess &&
             hipMemcpy(p->d_ranges, ranges.data(), ranges.size() * sizeof(int), hipMemcpyHostToDevice) == hipSuccess &&
             hipMalloc(reinterpret_cast<void**>(&p->d_clock), clock_bytes) == hipSuccess &&
             clear_clock(p) == hipSuccess;
        if (ok) {
            // the attribute belongs to the kernel, not to the plan: allow the
            // compute unit's whole LDS, so that no plan lowers another's limit
            const size_t lds = static_cast<size_t>(lds_cu);
            ok = (gdt == FC_F16 ? fc::prepare_resident_f16(sh, lds) : fc::prepare_resident_f32(sh, lds)) ==
                     hipSuccess &&
                 fc::prepare_resident_bcast(sh, lds) == hipSuccess;
        }
    }
    if (ok && !tiles.empty())
        ok = hipMemcpy(p->d_tiles, tiles.data(), tiles.size() * sizeof(Tile), hipMemcpyHostToDevice) == hipSuccess;
    if (ok)
        ok = hipMemcpy(p->d_mults, mults.data(), mults.size() * sizeof(float), hipMemcpyHostToDevice) ==
             hipSuccess;
    if (!ok) {
        free_plan(p);
        return FC_EHIP;
    }
    *plan = p;
    return FC_OK;
}

int fc_plan_create(fc_plan** plan, const fc_segment* segs, int nseg, int K, int gdt, int order) {
    return fc_plan_create_ex(plan, segs, nseg, K, gdt, order, nullptr);
}

void fc_plan_destroy(fc_plan* plan) { free_plan(plan); }

int fc_plan_query(const fc_plan* p, fc_plan_info* info) {
    if (!p || !info) return FC_EINVAL;
    info->K = p->K;
    info->nseg = static_cast<int>(p->segs.size());
    info->dtype = p->gdt;
    info->order = p->order;
    info->n_elems = p->n_elems;
    info->extent = p->extent;
    info->ntiles = p->ntiles;
    info->grid = p->grid;
    info->block_threads = p->shape.block;
    info->vecs_per_thread = p->shape.vecs;
    info->kchunk = p->shape.kchunk;
    info->schedule = p->res_one_launch ? FC_SCHED_RESIDENT_ONE_LAUNCH : p->schedule;
    info->scratch_bytes = p->d_sum ? p->extent * sizeof(float) : 0;
    info->k_waves = 1;
    info->lds_bytes = p->schedule == FC_SCHED_RESIDENT ? p->res_lds : 0;
    info->rounds = p->schedule == FC_SCHED_RESIDENT ? p->res_rounds : 0;
    if (p->schedule == FC_SCHED_RESIDENT) {
        // the launch of fc_step and fc_tree_reduce: one block of 16 waves per compute unit
        info->grid = p->res_grid;
        info->block_threads = 64 * fc::RESIDENT_WAVES;
    }
    return FC_OK;
}

static int fc_plan_balance_body(fc_plan* p, void* stream, float* xcd_rate, int n_rate) {
    if (!p || n_rate < 0 || (n_rate > 0 && !xcd_rate)) return FC_EINVAL;
    for (int i = 0; i < n_rate; ++i) xcd_rate[i] = 0.0f;
    if (p->schedule != FC_SCHED_RESIDENT || !p->res_record) return FC_OK;
    // no launch of this plan may still read the range table or write the
    // record: drain the given stream and the stream of the plan's last call
    // (neither may be capturing: a host wait would break the capture)
    const hipStream_t given = static_cast<hipStream_t>(stream);
    int crc = capture_check(given);
    if (!crc && p->have_last_stream && p->last_stream != given) crc = capture_check(p->last_stream);
    if (crc) return crc;
    if (hipStreamSynchronize(static_cast<hipStream_t>(stream)) != hipSuccess ||
        (p->have_last_stream && p->last_stream != static_cast<hipStream_t>(stream) &&
         hipStreamSynchronize(p->last_stream) != hipSuccess))
        return FC_EHIP;
    const int G = p->res_grid, R = p->res_rounds;
    std::vector<unsigned long long> c;
    std::vector<int> xcd;
    std::vector<double> rel_b;
    std::vector<int> ranges;
    try {
        c.resize(static_cast<size_t>(G) * fc::RESIDENT_CLOCK_WORDS);
        xcd.resize(static_cast<size_t>(G));
        rel_b.resize(static_cast<size_t>(G));
    } catch (const std::bad_alloc&) {
        return FC_ENOMEM;
    }
    if (hipMemcpy(c.data(), p->d_clock, c.size() * sizeof(unsigned long long), hipMemcpyDeviceToHost) != hipSuccess)
        return FC_EHIP;
    // tiles per tick of the reduce phase, per XCD, over every launch recorded
    constexpr int NX = 16;  // XCC_ID is 4 bits
    double tiles[NX] = {}, ticks[NX] = {};
    double all_tiles = 0.0, all_ticks = 0.0;
    for (int b = 0; b < G; ++b) {
        const unsigned long long* cb = &c[static_cast<size_t>(b) * fc::RESIDENT_CLOCK_WORDS];
        const int x = static_cast<int>(cb[2] & (NX - 1));
        xcd[b] = x;
        if (cb[0] > 0 && cb[1] > 0) {
            tiles[x] += static_cast<double>(cb[0]);
            ticks[x] += static_cast<double>(cb[1]);
            all_tiles += static_cast<double>(cb[0]);
            all_ticks += static_cast<double>(cb[1]);
        }
    }
    if (all_ticks <= 0.0) return FC_OK;  // nothing launched since the plan was made or last balanced
    const double mean = all_tiles / all_ticks;
    double rel[NX];
    for (int x = 0; x < NX; ++x) rel[x] = ticks[x] > 0.0 ? tiles[x] / ticks[x] / mean : 1.0;
    // shares proportional to the XCD's rate, drawn toward equal shares until
    // every block's tiles fit its LDS; equal shares always fit
    for (int b = 0; b < G; ++b) rel_b[b] = rel[xcd[b]];
    try {
        (void)fc::balanced_ranges(p->ntiles, R, G, rel_b, p->res_lds / p->res_slot + p->res_in_regs, ranges);
    } catch (const std::bad_alloc&) {
        return FC_ENOMEM;
    }
    if (hipMemcpy(p->d_ranges, ranges.data(), ranges.size() * sizeof(int), hipMemcpyHostToDevice) != hipSuccess ||
        clear_clock(p) != hipSuccess)
        return FC_EHIP;
    p->res_ranges.swap(ranges);
    for (int x = 0; x < n_rate && x < NX; ++x) xcd_rate[x] = ticks[x] > 0.0 ? static_cast<float>(rel[x]) : 0.0f;
    return FC_OK;
}

int fc_plan_set_timing(fc_plan* p, int enable) {
    if (!p) return FC_EINVAL;
    p->timing = enable != 0;
    return FC_OK;
}

static int fc_plan_read_timing_body(fc_plan* p, fc_timing* t) {
    if (!p || !t) return FC_EINVAL;
    std::memset(t, 0, sizeof(*t));
    int rc = FC_OK;
    for (auto& r : p->records) {
        float ms = 0.0f;
        if (rc == FC_OK && (hipEventSynchronize(r.b) != hipSuccess || hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess))
            rc = FC_EHIP;
        if (rc == FC_OK) {
            t->launches[r.kind] += 1;
            t->total_us[r.kind] += 1e3 * static_cast<double>(ms);
        }
        p->event_pool.push_back(r.a);
        p->event_pool.push_back(r.b);
    }
    p->records.clear();
    return rc;
}

namespace {

// Byte extent of a buffer of `elem` bytes per element covering the plan.
Span span_of(const fc_plan* p, const void* ptr, int elem, bool written, int id, bool replica) {
    const uintptr_t lo = reinterpret_cast<uintptr_t>(ptr);
    return Span{lo, lo + static_cast<uintptr_t>(p->extent) * elem, id, written, replica};
}

enum { ID_W = 1, ID_V, ID_OUT, ID_G, ID_SRC, ID_REPLICA0 = 16 };

int check_replicas(const fc_plan* p, const void* const* grads, Spans& spans) {
    if (!grads) return FC_EINVAL;
    for (int k = 0; k < p->K; ++k) {
        if (!grads[k]) return FC_EINVAL;
        if (!aligned16(grads[k])) return FC_EALIGN;
        spans.push(span_of(p, grads[k], p->sg, false, ID_REPLICA0 + k, true));
    }
    return FC_OK;
}

int check_dsts(const fc_plan* p, float* const* dst, Spans& spans) {
    for (int k = 0; k < p->K; ++k) {
        if (!dst[k]) return FC_EINVAL;
        if (!aligned16(dst[k])) return FC_EALIGN;
        spans.push(span_of(p, dst[k], 4, true, ID_REPLICA0 + p->K + k, false));
    }
    return FC_OK;
}

}  // namespace

static int fc_tree_reduce_body(fc_plan* p, const void* const* grads, float* out, void* stream) {
    if (!p || !out) return FC_EINVAL;
    if (!aligned16(out)) return FC_EALIGN;
    Spans spans;
    int rc = check_replicas(p, grads, spans);
    if (rc) return rc;
    spans.push(span_of(p, out, 4, true, ID_OUT, false));
    rc = check_aliasing(spans, ID_OUT, p->gdt == FC_F32);
    if (rc) return rc;
    if (p->ntiles == 0) return FC_OK;
    hipStream_t s = static_cast<hipStream_t>(stream);
    bool note = false;
    rc = order_after_last(p, s, note);
    if (rc) return rc;
    rc = update_table<const void*>(p, p->h_grads, p->grads_valid, p->d_grads, grads, s);
    if (rc == FC_OK) {
        fc::ReduceArgs a{};
        a.tiles = p->d_tiles;
        a.ntiles = p->ntiles;
        a.mults = p->d_mults;
        a.grads = p->d_grads;
        a.K = p->K;
        a.out = out;
        rc = launch(p, FC_KERNEL_REDUCE, s, [&] {
            return p->schedule == FC_SCHED_RESIDENT ? launch_resident(p, fc::MODE_REDUCE, a, s)
                                                    : launch_reduce(p->shape, fc::MODE_REDUCE, p->grid, a, s);
        });
    }
    if (note) note_stream(p, s);
    return rc;
}

static int fc_sgd_step_body(fc_plan* p, float* w, float* v, const float* g, float lr, float mu, float wd, int batch,
                void* stream) {
    if (!p || !w || !v || !g || batch < 1) return FC_EINVAL;
    if (!aligned16(w) || !aligned16(v) || !aligned16(g)) return FC_EALIGN;
    Spans spans;
    spans.push(span_of(p, w, 4, true, ID_W, false));
    spans.push(span_of(p, v, 4, true, ID_V, false));
    spans.push(span_of(p, g, 4, false, ID_G, false));
    int rc = check_aliasing(spans, -1, false);
    if (rc) return rc;
    if (p->ntiles == 0) return FC_OK;
    hipStream_t s = static_cast<hipStream_t>(stream);
    bool note = false;
    rc = order_after_last(p, s, note);
    if (rc) return rc;
    fc::SgdArgs a{};
    a.tiles = p->d_tiles;
    a.ntiles = p->ntiles;
    a.mults = p->d_mults;
    a.w = w;
    a.v = v;
    a.g = g;
    a.lr = lr;
    a.mu = mu;
    a.wd = wd;
    a.c = 1.0f / static_cast<float>(batch);
    rc = launch(p, FC_KERNEL_SGD, s, [&] { return fc::launch_sgd(p->shape, p->grid, a, s); });
    if (note) note_stream(p, s);
    return rc;
}

static int fc_broadcast_body(fc_plan* p, const float* src, float* const* dst, void* stream) {
    if (!p || !src || !dst) return FC_EINVAL;
    if (!aligned16(src)) return FC_EALIGN;
    Spans spans;
    spans.push(span_of(p, src, 4, false, ID_SRC, false));
    int rc = check_dsts(p, dst, spans);
    if (rc) return rc;
    rc = check_aliasing(spans, -1, false);
    if (rc) return rc;
    if (p->ntiles == 0) return FC_OK;
    hipStream_t s = static_cast<hipStream_t>(stream);
    bool note = false;
    rc = order_after_last(p, s, note);
    if (rc) return rc;
    rc = update_table<float*>(p, p->h_dst, p->dst_valid, p->d_dst, dst, s);
    if (rc == FC_OK) {
        fc::BcastArgs a{};
        a.tiles = p->d_tiles;
        a.ntiles = p->ntiles;
        a.src = src;
        a.dst = p->d_dst;
        a.K = p->K;
        rc = launch(p, FC_KERNEL_BCAST, s, [&] {
            if (p->schedule != FC_SCHED_RESIDENT) return fc::launch_bcast(p->shape, p->grid, a, s);
            // resident plans: the step's ranges, one launch per round, or
            // all rounds' ranges in one launch of grid x rounds blocks
            // (block b takes range b of the whole table)
            a.slots = p->res_lds / p->res_slot;
            const int per_launch = p->res_one_launch ? p->res_rounds : 1;
            for (int round = 0; round < p->res_rounds; round += per_launch) {
                a.ranges = p->d_ranges + static_cast<size_t>(round) * p->res_grid;
                const hipError_t e = fc::launch_resident_bcast(p->shape, p->res_grid * per_launch,
                                                               static_cast<size_t>(p->res_lds), a, s);
                if (e != hipSuccess) return e;
            }
            return hipSuccess;
        });
    }
    if (note) note_stream(p, s);
    return rc;
}

namespace {

// What fc_step and fc_step_noalloc check before they enqueue anything.
int check_step(const fc_plan* p, const void* const* grads, float* w, float* v, int batch, float* out,
               float* const* bcast_dst) {
    if (!p || !w || !v || batch < 1) return FC_EINVAL;
    if (!aligned16(w) || !aligned16(v) || (out && !aligned16(out))) return FC_EALIGN;
    Spans spans;
    int rc = check_replicas(p, grads, spans);
    if (rc) return rc;
    spans.push(span_of(p, w, 4, true, ID_W, false));
    spans.push(span_of(p, v, 4, true, ID_V, false));
    if (out) spans.push(span_of(p, out, 4, true, ID_OUT, false));
    if (bcast_dst) {
        rc = check_dsts(p, bcast_dst, spans);
        if (rc) return rc;
    }
    return check_aliasing(spans, out ? ID_OUT : -1, p->gdt == FC_F32);
}

// The replica table, and the destination table when broadcasting.
int update_step_tables(fc_plan* p, const void* const* grads, float* const* bcast_dst, hipStream_t s) {
    int rc = update_table<const void*>(p, p->h_grads, p->grads_valid, p->d_grads, grads, s);
    if (rc == FC_OK && bcast_dst) rc = update_table<float*>(p, p->h_dst, p->dst_valid, p->d_dst, bcast_dst, s);
    return rc;
}

// Two passes on the plan's tiles: the reduce kernel stores the raw sum into
// `sum`, then the SGD kernel updates w, v from it (and stores the broadcast
// copies).  `sh` is the launch shape of both passes.
int two_pass(fc_plan* p, const fc::Shape& sh, float* sum, float* w, float* v, float lr, float mu, float wd,
             float c, bool bcast, hipStream_t s, bool timed) {
    fc::ReduceArgs r{};
    r.tiles = p->d_tiles;
    r.ntiles = p->ntiles;
    r.mults = p->d_mults;
    r.grads = p->d_grads;
    r.K = p->K;
    r.out = sum;
    fc::SgdArgs g{};
    g.tiles = p->d_tiles;
    g.ntiles = p->ntiles;
    g.mults = p->d_mults;
    g.w = w;
    g.v = v;
    g.g = sum;
    g.dst = bcast ? p->d_dst : nullptr;
    g.K = p->K;
    g.lr = lr;
    g.mu = mu;
    g.wd = wd;
    g.c = c;
    if (!timed) {
        int rc = hip_rc(launch_reduce(sh, fc::MODE_REDUCE, p->grid, r, s));
        return rc ? rc : hip_rc(fc::launch_sgd(sh, p->grid, g, s));
    }
    int rc = launch(p, FC_KERNEL_REDUCE, s, [&] { return launch_reduce(sh, fc::MODE_REDUCE, p->grid, r, s); });
    if (rc == FC_OK) rc = launch(p, FC_KERNEL_SGD, s, [&] { return fc::launch_sgd(sh, p->grid, g, s); });
    return rc;
}

}  // namespace

static int fc_step_body(fc_plan* p, const void* const* grads, float* w, float* v, float lr, float mu, float wd, int batch,
            float* out, float* const* bcast_dst, void* stream) {
    int rc = check_step(p, grads, w, v, batch, out, bcast_dst);
    if (rc) return rc;
    if (p->ntiles == 0) return FC_OK;
    hipStream_t s = static_cast<hipStream_t>(stream);
    bool note = false;
    rc = order_after_last(p, s, note);
    if (rc) return rc;
    rc = update_step_tables(p, grads, bcast_dst, s);
    const float c = 1.0f / static_cast<float>(batch);
    if (rc == FC_OK && p->schedule == FC_SCHED_TWO_PASS) {
        // pass 1: raw sum into `out` (or the plan's scratch); pass 2: update (+ broadcast)
        rc = two_pass(p, p->shape, out ? out : p->d_sum, w, v, lr, mu, wd, c, bcast_dst != nullptr, s, true);
    } else if (rc == FC_OK) {
        fc::ReduceArgs a{};
        a.tiles = p->d_tiles;
        a.ntiles = p->ntiles;
        a.mults = p->d_mults;
        a.grads = p->d_grads;
        a.K = p->K;
        a.w = w;
        a.v = v;
        a.out = out;
        a.dst = bcast_dst ? p->d_dst : nullptr;
        a.lr = lr;
        a.mu = mu;
        a.wd = wd;
        a.c = c;
        rc = launch(p, FC_KERNEL_STEP, s, [&] {
            return p->schedule == FC_SCHED_RESIDENT ? launch_resident(p, fc::MODE_STEP, a, s)
                                                    : launch_reduce(p->shape, fc::MODE_STEP, p->grid, a, s);
        });
    }
    if (note) note_stream(p, s);
    return rc;
}

// fc_step's two-pass schedule with the raw sum in the library's fixed device
// array (fc_update.hip) instead of memory the plan owns; it allocates
// nothing, on the device or on the host.
static int fc_step_noalloc_body(fc_plan* p, const void* const* grads, float* w, float* v, float lr, float mu,
                                float wd, int batch, float* out, float* const* bcast_dst, void* stream) {
    int rc = check_step(p, grads, w, v, batch, out, bcast_dst);
    if (rc) return rc;
    if (!out && p->extent > static_cast<uint64_t>(FC_NOALLOC_MAX_ELEMS)) return FC_ESIZE;
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return FC_EHIP;
    if (dev != p->device) return FC_EINVAL;
    if (p->ntiles == 0) return FC_OK;
    // both passes run on the plan's tiles (block * vecs lane-vectors each);
    // a resident plan's batch of 4 replicas has no reduce-kernel instance,
    // so its reduce pass loads batches of 8 (the association does not depend
    // on the batch)
    fc::Shape sh = p->shape;
    if (!fc::compiled_pair(sh.vecs, sh.kchunk)) {
        sh.kchunk = 8;
        sh.maxd = bit_length(p->K / sh.kchunk);
    }
    float* sum = out;
    if (!sum) {
        rc = hip_rc(fc::noalloc_scratch(dev, &sum));
        if (rc) return rc;
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    bool note = false;
    rc = order_after_last(p, s, note);
    if (rc) return rc;
    rc = update_step_tables(p, grads, bcast_dst, s);
    if (rc == FC_OK)
        rc = two_pass(p, sh, sum, w, v, lr, mu, wd, 1.0f / static_cast<float>(batch), bcast_dst != nullptr, s,
                      false);
    if (note) note_stream(p, s);
    return rc;
}

uint64_t fc_read_probe_blocks(uint64_t bytes) { return fc::read_probe_blocks(bytes); }

int fc_read_probe(const void* src, uint64_t bytes, float* out, void* stream) {
    if (!src || !out || bytes == 0 || bytes % 16) return FC_EINVAL;
    if (!aligned16(src) || (reinterpret_cast<uintptr_t>(out) & 3u)) return FC_EALIGN;
    // one block per 16 KiB; the grid's x dimension is 32 bits
    if (fc::read_probe_blocks(bytes) > 0x7fffffffu) return FC_EINVAL;
    return hip_rc(fc::launch_read_probe(src, bytes, out, static_cast<hipStream_t>(stream)));
}

int fc_lr_at(const fc_lr_policy* pol, int64_t iter, int batch, float* lr) {
    if (!pol || !lr || iter < 0 || batch < 1) return FC_EINVAL;
    if (!(pol->base_lr >= 0.0) || pol->base_batch < 0) return FC_EINVAL;
    double factor = 1.0;
    switch (pol->kind) {
        case FC_LR_FIXED:
            break;
        case FC_LR_STEP:
            if (pol->stepsize < 1 || !(pol->gamma > 0.0)) return FC_EINVAL;
            factor = std::pow(pol->gamma, static_cast<double>(iter / pol->stepsize));
            break;
        case FC_LR_POLY:
            if (pol->max_iter < 1 || iter > pol->max_iter || !(pol->power >= 0.0)) return FC_EINVAL;
            factor = std::pow(1.0 - static_cast<double>(iter) / static_cast<double>(pol->max_iter), pol->power);
            break;
        default:
            return FC_EINVAL;
    }
    const double scale =
        pol->base_batch > 0 ? static_cast<double>(batch) / static_cast<double>(pol->base_batch) : 1.0;
    *lr = static_cast<float>(pol->base_lr * scale * factor);
    return FC_OK;
}

int fc_train(fc_plan* p, const void* const* grads, float* w, float* v, const fc_lr_policy* policy,
             int64_t first_iter, int64_t n_iters, float mu, float wd, int batch, void* stream) {
    if (!p || !policy || first_iter < 0 || n_iters < 0) return FC_EINVAL;
    float lr = 0.0f;
    // check the whole schedule before enqueuing anything
    if (n_iters > 0) {
        int rc = fc_lr_at(policy, first_iter + n_iters - 1, batch, &lr);
        if (rc) return rc;
    }
    for (int64_t it = first_iter; it < first_iter + n_iters; ++it) {
        int rc = fc_lr_at(policy, it, batch, &lr);
        if (rc == FC_OK) rc = fc_step(p, grads, w, v, lr, mu, wd, batch, nullptr, nullptr, stream);
        if (rc) return rc;
    }
    return FC_OK;
}

int fc_plan_read_timing(fc_plan* p, fc_timing* t) {
    return guarded([&] { return fc_plan_read_timing_body(p, t); });
}

int fc_tree_reduce(fc_plan* p, const void* const* grads, float* out, void* stream) {
    return guarded([&] { return fc_tree_reduce_body(p, grads, out, stream); });
}

int fc_sgd_step(fc_plan* p, float* w, float* v, const float* g, float lr, float mu, float wd, int batch,
                void* stream) {
    return guarded([&] { return fc_sgd_step_body(p, w, v, g, lr, mu, wd, batch, stream); });
}

int fc_broadcast(fc_plan* p, const float* src, float* const* dst, void* stream) {
    return guarded([&] { return fc_broadcast_body(p, src, dst, stream); });
}

int fc_step(fc_plan* p, const void* const* grads, float* w, float* v, float lr, float mu, float wd, int batch,
            float* out, float* const* bcast_dst, void* stream) {
    return guarded([&] { return fc_step_body(p, grads, w, v, lr, mu, wd, batch, out, bcast_dst, stream); });
}

int fc_step_noalloc(fc_plan* p, const void* const* grads, float* w, float* v, float lr, float mu, float wd,
                    int batch, float* out, float* const* bcast_dst, void* stream) {
    // no try/catch here: nothing on this path allocates or throws
    return fc_step_noalloc_body(p, grads, w, v, lr, mu, wd, batch, out, bcast_dst, stream);
}

int fc_plan_balance(fc_plan* p, void* stream, float* xcd_rate, int n_rate) {
    return guarded([&] { return fc_plan_balance_body(p, stream, xcd_rate, n_rate); });
}

}  // extern "C"

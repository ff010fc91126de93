"""HIP path vs the oracle, bit for bit, through the C ABI.

Sizes: ragged random segment tables of a few tens of thousands of elements
(several tiles per segment, lengths that are not multiples of the vector
width, tiny segments) so the oracle finishes in well under a second per case.
Tolerance: none -- the reduced sums and the SGD update are compared bit for
bit (NaN compared as NaN), because both sides perform the same fp32
operations in the same order with no contraction.
"""
import numpy as np
import pytest

from gpu_cases import LR, MU, WD, alloc_len, host_replicas, run_reduce, run_steps, same_bits, to_dev
import oracle
from workloads import gen

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def fc(device):
    import paper_1511_00175_amd as m
    return m


def table(seed, dtype, nseg=9, max_len=5000):
    rng = np.random.default_rng(seed)
    vec = 4  # offsets: multiples of 4 elements for both storage types
    rows, _ = gen.random_table(rng, nseg, max_len, vec)
    # a tiny segment, one exactly one default tile long, one a tile plus one
    off = rows[-1][0] + rows[-1][1]
    off = (off + vec - 1) // vec * vec
    for n in (3, 256 * vec, 256 * vec + 1, 16):
        rows.append((off, n, 1.0, 1.0))
        off = (off + n + 63) // 64 * 64
    return rows


KS = [1, 2, 3, 4, 5, 7, 8, 9, 15, 16, 17, 31, 32, 33, 64, 100, 128]


@pytest.mark.parametrize("dtype", ["f32", "f16"])
@pytest.mark.parametrize("order", ["tree", "linear"])
@pytest.mark.parametrize("K", KS)
def test_reduce_matches_oracle(fc, K, order, dtype):
    segs = table(1000 + K, dtype)
    bad, _, _ = run_reduce(fc, segs, K, dtype, order, np.random.default_rng(K))
    assert bad == 0


@pytest.mark.parametrize("dtype", ["f32", "f16"])
@pytest.mark.parametrize("order", ["tree", "linear"])
@pytest.mark.parametrize("K", KS)
def test_step_matches_oracle(fc, K, order, dtype):
    segs = [(o, n, lm, dm) for (o, n, lm, dm) in table(2000 + K, dtype)]
    # non-uniform multipliers on some segments (Caffe-style bias settings)
    segs = [(o, n, 2.0, 0.0) if i % 3 == 1 else (o, n, lm, dm) for i, (o, n, lm, dm) in enumerate(segs)]
    assert run_steps(fc, segs, K, dtype, order, np.random.default_rng(K), steps=3) == 0


@pytest.mark.parametrize("dtype", ["f32", "f16"])
@pytest.mark.parametrize("order", ["tree", "linear"])
@pytest.mark.parametrize("K", [1, 3, 8, 32, 100])
def test_step_with_sum_and_broadcast(fc, K, order, dtype):
    segs = table(3000 + K, dtype, nseg=5, max_len=3000)
    assert run_steps(fc, segs, K, dtype, order, np.random.default_rng(K), steps=2, with_out=True,
                     with_bcast=True) == 0


@pytest.mark.parametrize("dtype", ["f32", "f16"])
@pytest.mark.parametrize("order", ["tree", "linear"])
@pytest.mark.parametrize("K", [1, 2, 5, 16, 33])
def test_special_values(fc, K, order, dtype):
    """Signed zeros, subnormals of the storage type, infinities and NaN."""
    segs = table(4000 + K, dtype, nseg=4, max_len=2000)
    bad, _, _ = run_reduce(fc, segs, K, dtype, order, np.random.default_rng(K), special=True)
    assert bad == 0
    assert run_steps(fc, segs, K, dtype, order, np.random.default_rng(K), steps=2, special=True) == 0


@pytest.mark.parametrize("K", [256, 1000, 1024])
def test_many_workers(fc, K):
    """K beyond 31 chunks uses the deeper pending-subtree stack, in the
    default schedule and in the resident kernel (its depth-7 instances)."""
    segs = [(0, 1000, 1, 1), (1024, 37, 1, 1), (1088, 8, 1, 1)]
    for opts in (None, dict(schedule=3)):
        for dtype in ("f32", "f16"):
            for order in ("tree", "linear"):
                bad, _, _ = run_reduce(fc, segs, K, dtype, order, np.random.default_rng(K), opts=opts)
                assert bad == 0, (dtype, order, opts)
                assert run_steps(fc, segs, K, dtype, order, np.random.default_rng(K), steps=1, opts=opts,
                                 with_out=True, with_bcast=K == 256) == 0, (dtype, order, opts)


def test_fp16_widening_exhaustive(fc):
    """All 65536 binary16 patterns as one K=1 replica: the sum is the widened
    value (numpy's float16->float32 conversion, a library routine)."""
    import torch
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    ref = bits.view(np.float16).astype(np.float32)
    plan = fc.Plan([(0, 1 << 16)], 1, "f16", "tree")
    out = torch.zeros(1 << 16, device="cuda")
    plan.tree_reduce([to_dev(bits.view(np.float16))], out)
    assert same_bits(out.cpu().numpy(), ref) == 0


PAIRS = [(1, 8), (1, 16), (2, 8), (2, 16), (4, 2), (4, 4), (4, 8)]
SHAPES = [dict(block_threads=b, vecs_per_thread=u, kchunk=c) for b in (64, 128, 256) for u, c in PAIRS]
SHAPES += [dict(schedule=2), dict(schedule=2, block_threads=256, vecs_per_thread=2, kchunk=8, max_blocks=5)]
SHAPES += [dict(schedule=3), dict(schedule=3, max_blocks=7), dict(schedule=3, max_blocks=1)]

FP16_PAIR_OPTS = [None, dict(schedule=2), dict(schedule=3), dict(schedule=3, vecs_per_thread=2, kchunk=4)]
FP16_PAIR_OPTS += [dict(block_threads=256, vecs_per_thread=u, kchunk=c) for u, c in PAIRS]


def fp16_pattern_replicas(K, m, pos):
    """K fp16 replicas of m elements: every binary16 pattern in leaf pos, a
    partner pattern (an odd multiplier makes the map a bijection of the
    16-bit patterns) in leaf pos + 1 and +0 elsewhere; pos None: every leaf
    holds its own bijection of the patterns."""
    n = 1 << 16
    bits = np.arange(n, dtype=np.uint32)
    reps = np.zeros((K, m), np.uint16)
    if pos is None:
        for k in range(K):
            reps[k, :n] = (bits * np.uint32(2 * k + 40503) + np.uint32(977 * k)) & 0xFFFF
    else:
        reps[pos, :n] = bits
        reps[pos + 1, :n] = (bits * np.uint32(40503) + np.uint32(12345)) & 0xFFFF
    return reps.view(np.float16)


@pytest.mark.parametrize("order", ["tree", "linear"])
@pytest.mark.parametrize("K, positions", [(16, (0, 2, 4, 6, 8, 10, 12, 14, None)), (23, (0, 6, 14, 16, 21, None))])
def test_fp16_pair_sums_exhaustive(fc, K, positions, order):
    """Sums of widened fp16 leaves: every binary16 pattern -- subnormals,
    signed zeros, infinities, NaNs -- meets a partner pattern in every leaf
    position of a chunk and of the remainder (K = 23), in both orders, for
    every schedule and compiled fp16 shape; the raw sums and one step match
    the oracle bit for bit."""
    import torch
    segs = [(0, 1 << 16, 1.0, 1.0)]
    m = alloc_len(segs)
    w = np.random.default_rng(K).standard_normal(m, dtype=np.float32) * np.float32(0.05)
    for pos in positions:
        reps = fp16_pattern_replicas(K, m, pos)
        expect = oracle.tree_reduce(segs, list(reps), order=order, out=np.zeros(m, np.float32))
        w1, v1, _, _ = oracle.step(segs, list(reps), w, np.zeros(m, np.float32), LR, MU, WD, 256, order=order)
        reps_d = to_dev(reps)
        for opts in FP16_PAIR_OPTS:
            plan = fc.Plan(segs, K, "f16", order, **(opts or {}))
            out = torch.zeros(m, device="cuda")
            plan.tree_reduce(reps_d, out)
            assert same_bits(out.cpu().numpy(), expect) == 0, (pos, opts)
            if opts is None or "schedule" in opts:
                w_d, v_d = to_dev(w), torch.zeros(m, device="cuda")
                plan.step(reps_d, w_d, v_d, LR, MU, WD, 256)
                assert same_bits(w_d.cpu().numpy(), w1) + same_bits(v_d.cpu().numpy(), v1) == 0, (pos, opts)
            plan.close()


@pytest.mark.parametrize("dtype", ["f32", "f16"])
@pytest.mark.parametrize("order", ["tree", "linear"])
def test_launch_shape_invariance(fc, dtype, order):
    """Identical bits for every launch shape (and a capped grid that makes
    blocks loop over tiles) -- the association never depends on it."""
    segs = table(5000, dtype)
    K = 37
    ref = None
    for opts in SHAPES + [dict(max_blocks=7), dict(max_blocks=1, vecs_per_thread=2, kchunk=16)]:
        bad, got, expect = run_reduce(fc, segs, K, dtype, order, np.random.default_rng(5), opts=opts)
        assert bad == 0, opts
        if ref is None:
            ref = got
        assert same_bits(got, ref) == 0
        assert run_steps(fc, segs, K, dtype, order, np.random.default_rng(6), steps=1, opts=opts) == 0, opts


@pytest.mark.parametrize("dtype", ["f32", "f16"])
@pytest.mark.parametrize("order", ["tree", "linear"])
@pytest.mark.parametrize("schedule", [1, 2, 3, 4])
@pytest.mark.parametrize("K", [3, 64, 130])
def test_schedules_match_oracle(fc, K, schedule, order, dtype):
    """fc_step in one fused pass, in two passes (raw sum, then update) and
    resident (one launch per round, or every round in one launch), with and
    without the raw sum and the broadcast, over chained steps, in both
    orders."""
    segs = table(9000 + K, dtype, nseg=5, max_len=3000)
    rng = np.random.default_rng(K + schedule)
    for with_out, with_bcast in ((False, False), (True, False), (False, True), (True, True)):
        assert run_steps(fc, segs, K, dtype, order, rng, steps=2, opts=dict(schedule=schedule),
                         with_out=with_out, with_bcast=with_bcast) == 0, (with_out, with_bcast)


def test_schedule_resolution(fc):
    """AUTO keeps steps of less than 64 MiB on the fused kernel (two passes
    when a parameter's replicas exceed 256 bytes); above that it takes the
    resident schedule when every block's share of tiles fits a compute
    unit's LDS; otherwise two passes when a parameter's replicas exceed 256
    bytes, only then with a raw-sum scratch buffer."""
    import torch
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    small = [(0, 1000, 1, 1), (1024, 5, 1, 1)]
    for K, dtype, sched in ((1, "f32", 1), (64, "f32", 1), (65, "f32", 2), (1024, "f32", 2), (128, "f16", 1),
                            (129, "f16", 2)):
        info = fc.Plan(small, K, dtype, "tree").info()
        assert (info.schedule, info.rounds) == (sched, 0), (K, dtype)
    # a batch alone names single-vector resident tiles, also where the
    # default would take two vectors (fp32, K <= 16)
    info = fc.Plan(small, 8, "f32", "tree", schedule=3, kchunk=16).info()
    assert (info.vecs_per_thread, info.kchunk) == (1, 16)
    assert run_steps(fc, small, 8, "f32", "tree", np.random.default_rng(4), steps=2,
                     opts=dict(schedule=3, kchunk=16)) == 0
    # 2^20 x K=4 fp32 (32 MiB of replicas + 16 MiB of w, v): fused; K=16 (80 MiB): resident
    assert fc.Plan([(0, 1 << 20, 1, 1)], 4, "f32", "tree").info().schedule == 1
    assert fc.Plan([(0, 1 << 20, 1, 1)], 16, "f32", "tree").info().schedule == 3
    for K, dtype in ((1, "f32"), (16, "f32"), (17, "f32"), (64, "f32"), (1024, "f32"), (129, "f16")):
        info = fc.Plan(small, K, dtype, "tree", schedule=3).info()
        assert (info.schedule, info.scratch_bytes, info.rounds) == (3, 0, 1), (K, dtype)
        if dtype == "f32" and K <= 16:
            # tiles of 2 vectors per lane, batches of 4: 2 tiles of 512 elements
            # (the second of 488), then the 5-element segment's vector and its
            # tail tile; one round either way, so no register-held tiles: LDS
            # for the 4 tiles a block could be given, 2 KiB each
            assert (info.block_threads, info.vecs_per_thread, info.kchunk, info.k_waves) == (1024, 2, 4, 1)
            assert (info.ntiles, info.grid, info.lds_bytes) == (4, 4, 4 * 2048)
        else:
            assert (info.block_threads, info.vecs_per_thread, info.kchunk, info.k_waves) == (1024, 1, 16, 1)
            # 3 tiles of 256 elements and one of 232, then the 5-element segment's
            # vector and its tail tile: one tile per block; LDS for the 6 tiles a
            # block could be given (fc_plan_balance), 1 KiB each
            assert (info.ntiles, info.grid, info.lds_bytes) == (6, 6, 6 * 1024)
    # fp32 K=8: tiles of 512 elements, 144 per block and round (80 in 160 KiB
    # of LDS, 4 in the registers of each of the 16 waves)
    fits = [(0, cus * 144 * 512, 1, 1)]
    big = [(0, cus * 144 * 512 + 4, 1, 1)]
    info = fc.Plan(fits, 8, "f32", "tree").info()
    assert (info.schedule, info.rounds, info.lds_bytes, info.grid) == (3, 1, 160 * 1024, cus)
    for K, dtype, two in ((64, "f32", False), (65, "f32", True), (128, "f16", False), (129, "f16", True)):
        p = fc.Plan(big, K, dtype, "tree", k_waves=1)
        info = p.info()
        assert info.schedule == (2 if two else 1), (K, dtype)
        assert info.scratch_bytes == (4 * big[0][1] if two else 0)
        p.close()
    # without a launch shape, plans of several rounds are resident when a
    # parameter's replicas take at least 48 bytes (400 tiles of 256 per CU
    # exceed a round with any register-held tiles)
    several = [(0, cus * 400 * 256, 1, 1)]
    for K, dtype, sched in ((11, "f32", 1), (12, "f32", 3), (23, "f16", 1), (24, "f16", 3), (130, "f32", 3)):
        p = fc.Plan(several, K, dtype, "tree")
        assert p.info().rounds >= 2 or sched == 1, (K, dtype)
        assert p.info().schedule == sched, (K, dtype)
        p.close()
    assert fc.Plan(small, 128, "f32", "tree", schedule=1).info().scratch_bytes == 0
    # an explicit launch shape keeps AUTO off the resident kernel; a plan that
    # needs more than one round is resident only when asked for
    assert fc.Plan(small, 8, "f32", "tree", block_threads=64).info().schedule == 1
    assert fc.Plan(big, 8, "f32", "tree").info().schedule == 1
    assert fc.Plan(big, 64, "f32", "tree", block_threads=64).info().schedule == 1
    assert fc.Plan(big, 65, "f32", "tree", block_threads=64).info().schedule == 2
    info = fc.Plan(big, 8, "f32", "tree", schedule=3).info()
    assert (info.schedule, info.rounds, info.lds_bytes) == (3, 2, 160 * 1024)
    # 1 vector and batches of 16 (fp32, K > 16): 160 tiles of 256 per block
    # and round, all in LDS
    info = fc.Plan([(0, cus * 160 * 256, 1, 1)], 20, "f32", "tree").info()
    assert (info.schedule, info.rounds, info.lds_bytes, info.vecs_per_thread) == (3, 1, 160 * 1024, 1)
    info = fc.Plan([(0, cus * 160 * 256 + 4, 1, 1)], 20, "f32", "tree").info()
    assert (info.schedule, info.rounds, info.lds_bytes) == (3, 2, 160 * 1024)


def test_timing_records_every_launch(fc):
    import torch
    segs = [(0, 5000, 1, 1)]
    K = 130
    reps = torch.randn((K, 5120), device="cuda")
    w, v, g = (torch.zeros(5120, device="cuda") for _ in range(3))
    for schedule in (1, 2, 3):
        plan = fc.Plan(segs, K, "f32", "tree", schedule=schedule)
        plan.set_timing(True)
        for _ in range(3):
            plan.step(reps, w, v, 0.1, 0.9, 0.0, 64)
        plan.tree_reduce(reps, g)
        t = plan.read_timing()
        if schedule in (1, 3):
            assert t["step"][0] == 3 and t["reduce"][0] == 1 and t["sgd"][0] == 0
        else:
            assert t["step"][0] == 0 and t["reduce"][0] == 4 and t["sgd"][0] == 3
        assert all(us > 0 for n, us in t.values() if n)
        assert all(n == 0 for n, _ in plan.read_timing().values())
        plan.set_timing(False)
        plan.step(reps, w, v, 0.1, 0.9, 0.0, 64)
        assert all(n == 0 for n, _ in plan.read_timing().values())
        plan.close()


def test_fused_equals_composed(fc):
    """fc_step == fc_tree_reduce, then fc_sgd_step, then fc_broadcast of w'."""
    import torch
    rng = np.random.default_rng(7)
    segs = table(7000, "f32")
    K = 24
    n = max(o + ln for o, ln, _, _ in segs) + 64
    reps = to_dev((rng.standard_normal((K, n)) * 1e-2).astype(np.float32))
    w0 = to_dev((rng.standard_normal(n) * 0.05).astype(np.float32))
    v0 = to_dev((rng.standard_normal(n) * 1e-3).astype(np.float32))
    plan = fc.Plan(segs, K, "f32", "tree")
    w1, v1, out1 = w0.clone(), v0.clone(), torch.zeros(n, device="cuda")
    d1 = torch.zeros((K, n), device="cuda")
    plan.step(reps, w1, v1, 0.02, 0.9, 1e-4, 128, out=out1, bcast=d1)
    w2, v2, g = w0.clone(), v0.clone(), torch.zeros(n, device="cuda")
    d2 = torch.zeros((K, n), device="cuda")
    plan.tree_reduce(reps, g)
    plan.sgd_step(w2, v2, g, 0.02, 0.9, 1e-4, 128)
    plan.broadcast(w2, d2)
    torch.cuda.synchronize()
    for a, b in ((w1, w2), (v1, v2), (out1, g), (d1, d2)):
        assert same_bits(a.cpu().numpy(), b.cpu().numpy()) == 0


@pytest.mark.parametrize("dtype", ["f32", "f16"])
@pytest.mark.parametrize("schedule,max_blocks,vecs", [(0, 0, 0), (1, 0, 0), (2, 0, 0), (3, 0, 1), (3, 0, 2),
                                                      (3, 1, 1), (3, 1, 2), (3, 2, 1), (4, 1, 1), (4, 2, 2)])
@pytest.mark.parametrize("K", [1, 5, 40])
def test_broadcast_matches_oracle(fc, K, schedule, max_blocks, vecs, dtype):
    """fc_broadcast on each schedule's tile map: on resident plans one
    persistent block per CU stages its range of the source in LDS and stores
    it one destination at a time (one round, or many with few blocks, one
    launch per round or all rounds' blocks in one launch); on the others one
    block per tile.  Every destination gets the source's bits on
    every segment element (special values included) and keeps its fill
    value elsewhere; the replica type only changes the plan's tile map."""
    import torch
    segs = table(15000 + K, dtype, nseg=8, max_len=60000)  # 248-354 K elements: 970+ tiles of 256
    n = alloc_len(segs)
    rng = np.random.default_rng(K * 31 + schedule * 7 + max_blocks)
    src = host_replicas(rng, 1, n, np.float32, special=True)[0]
    expect = oracle.broadcast(segs, src, [np.full(n, -2.0, np.float32) for _ in range(K)])
    opts = dict(schedule=schedule, max_blocks=max_blocks) if schedule else {}
    if vecs:
        opts["vecs_per_thread"] = vecs
    plan = fc.Plan(segs, K, dtype, "tree", **opts)
    if schedule in (3, 4) and max_blocks:
        assert (plan.info().schedule, plan.info().rounds > 1) == (schedule, True)
    dst = torch.full((K, n), -2.0, device="cuda")
    plan.broadcast(to_dev(src), dst)
    torch.cuda.synchronize()
    got = dst.cpu().numpy()
    plan.close()
    assert sum(same_bits(got[k], expect[k]) for k in range(K)) == 0


def test_repeatable(fc):
    """The same inputs give the same bits on every run (FAQ 6: no
    nondeterministic techniques)."""
    segs = table(8000, "f32")
    r1 = run_reduce(fc, segs, 64, "f32", "tree", np.random.default_rng(3))[1]
    for _ in range(3):
        r2 = run_reduce(fc, segs, 64, "f32", "tree", np.random.default_rng(3))[1]
        assert same_bits(r1, r2) == 0


def test_out_may_be_a_replica(fc):
    """out == grads[k] exactly is allowed for fp32 replicas and gives the sum."""
    import oracle
    import torch
    rng = np.random.default_rng(9)
    segs = [(0, 4000, 1, 1), (4096, 77, 1, 1)]
    K, n = 6, 4224
    reps = (rng.standard_normal((K, n))).astype(np.float32)
    expect = oracle.tree_reduce(segs, list(reps), out=reps[2].copy())
    plan = fc.Plan(segs, K, "f32", "tree")
    rd = to_dev(reps)
    plan.tree_reduce(rd, rd[2])
    torch.cuda.synchronize()
    assert same_bits(rd[2].cpu().numpy(), expect) == 0


def test_argument_errors_need_a_plan(fc):
    import torch
    f = fc._fc
    plan = fc.Plan([(0, 1000, 1, 1)], 4, "f32", "tree")
    buf = torch.zeros(8192, device="cuda")
    reps = [buf[i * 1024:].data_ptr() for i in range(4)]
    out = torch.zeros(1024, device="cuda")
    w = torch.zeros(1024, device="cuda")
    v = torch.zeros(1024, device="cuda")
    s = torch.cuda.current_stream().cuda_stream
    h = plan.handle
    # misaligned pointers
    assert f.fc_tree_reduce(h, reps, out.data_ptr() + 4, s) == f.FC_EALIGN
    assert f.fc_tree_reduce(h, [reps[0] + 8] + reps[1:], out.data_ptr(), s) == f.FC_EALIGN
    # null replica
    assert f.fc_tree_reduce(h, [0] + reps[1:], out.data_ptr(), s) == f.FC_EINVAL
    # out partially overlapping a replica
    assert f.fc_tree_reduce(h, reps, reps[1] + 16, s) == f.FC_EALIAS
    # w == v, v overlapping g
    assert f.fc_sgd_step(h, w.data_ptr(), w.data_ptr(), out.data_ptr(), 0.1, 0.9, 0.0, 1, s) == f.FC_EALIAS
    assert f.fc_sgd_step(h, w.data_ptr(), out.data_ptr() + 16, out.data_ptr(), 0.1, 0.9, 0.0, 1, s) == f.FC_EALIAS
    assert f.fc_sgd_step(h, w.data_ptr(), v.data_ptr(), out.data_ptr(), 0.1, 0.9, 0.0, 0, s) == f.FC_EINVAL
    # broadcast destinations overlapping each other or the source
    dst = [buf[4096 + 1024 * i:].data_ptr() for i in range(4)]
    assert f.fc_broadcast(h, out.data_ptr(), dst[:3] + [dst[2]], s) == f.FC_EALIAS
    assert f.fc_broadcast(h, dst[0], dst, s) == f.FC_EALIAS
    # a broadcast destination overlapping w
    assert f.fc_step(h, reps, w.data_ptr(), v.data_ptr(), 0.1, 0.9, 0.0, 1, None, dst[:3] + [w.data_ptr()],
                     s) == f.FC_EALIAS
    # w inside a replica; v ending inside w; the raw sum exactly on w
    assert f.fc_step(h, reps, reps[2] + 64, v.data_ptr(), 0.1, 0.9, 0.0, 1, None, None, s) == f.FC_EALIAS
    assert f.fc_step(h, reps, w.data_ptr(), w.data_ptr() - 16, 0.1, 0.9, 0.0, 1, None, None, s) == f.FC_EALIAS
    assert f.fc_step(h, reps, w.data_ptr(), v.data_ptr(), 0.1, 0.9, 0.0, 1, w.data_ptr(), None, s) == f.FC_EALIAS
    torch.cuda.synchronize()
    # nothing was written by the rejected calls
    assert float(out.abs().sum()) == 0.0 and float(w.abs().sum()) == 0.0
    # read-only buffers may overlap: every replica the same pointer is a valid call
    assert f.fc_tree_reduce(h, [reps[0]] * 4, out.data_ptr(), s) == f.FC_OK
    torch.cuda.synchronize()


def test_empty_and_zero_length(fc):
    import torch
    plan = fc.Plan([], 3, "f32", "tree")
    assert plan.info().ntiles == 0
    x = torch.zeros((3, 64), device="cuda")
    w, v = torch.ones(64, device="cuda"), torch.ones(64, device="cuda")
    plan.step(x, w, v, 0.1, 0.9, 0.1, 1)
    plan.tree_reduce(x, w)
    torch.cuda.synchronize()
    assert float(w.sum()) == 64.0
    segs = [(0, 0, 1, 1), (8, 5, 1, 1), (16, 0, 1, 1)]
    bad, got, _ = run_reduce(fc, segs, 3, "f32", "tree", np.random.default_rng(1))
    assert bad == 0


@pytest.mark.parametrize("K,dtype,schedule,max_blocks", [(4, "f32", 1, 0), (130, "f32", 2, 0), (16, "f16", 1, 0),
                                                         (128, "f32", 0, 0), (40, "f32", 3, 1), (40, "f32", 4, 1)])
def test_graph_capture_replays(fc, K, dtype, schedule, max_blocks):
    """A step whose pointer tables are already on the device, called on the
    stream it last ran on, enqueues kernel launches only, so it can be
    captured in a HIP graph.  Every replay (with eager steps and
    synchronizations in between) gives the bits of an eager twin plan."""
    import torch
    segs = table(13000 + K, dtype, nseg=4, max_len=3000)
    if max_blocks:  # one block of 160 tile slots: the resident step takes several rounds (launches)
        segs = segs + [(segs[-1][0] + segs[-1][1] + 64 - (segs[-1][0] + segs[-1][1]) % 64, 45000, 1.0, 1.0)]
    n = alloc_len(segs)
    rng = np.random.default_rng(K)
    npdt = np.float16 if dtype == "f16" else np.float32
    reps = to_dev(host_replicas(rng, K, n, npdt, scale=0.01))
    w0 = (rng.standard_normal(n, dtype=np.float32) * np.float32(0.05))
    wa, va = to_dev(w0), torch.zeros(n, device="cuda")
    wb, vb = to_dev(w0), torch.zeros(n, device="cuda")
    pa = fc.Plan(segs, K, dtype, "tree", schedule=schedule, max_blocks=max_blocks)
    pb = fc.Plan(segs, K, dtype, "tree", schedule=schedule, max_blocks=max_blocks)
    if max_blocks:
        assert pa.info().rounds >= 2
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        pa.step(reps, wa, va, LR, MU, WD, 256)
    s.synchronize()
    pb.step(reps, wb, vb, LR, MU, WD, 256)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        pa.step(reps, wa, va, LR, MU, WD, 256)
    for _ in range(3):
        g.replay()
        torch.cuda.synchronize()
        pb.step(reps, wb, vb, LR, MU, WD, 256)
        torch.cuda.synchronize()
        assert same_bits(wa.cpu().numpy(), wb.cpu().numpy()) == 0
        assert same_bits(va.cpu().numpy(), vb.cpu().numpy()) == 0
    pa.close()
    pb.close()


def test_calls_default_to_torchs_current_stream(fc):
    """Without a stream argument a call runs on torch's current stream of the
    current device, also inside a stream context."""
    import torch
    from paper_1511_00175_amd import _stream
    assert _stream(None) == torch.cuda.current_stream().cuda_stream
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        assert _stream(None) == s.cuda_stream == torch.cuda.current_stream().cuda_stream
    assert _stream(None) == torch.cuda.current_stream().cuda_stream
    assert _stream(s) == s.cuda_stream and _stream(s.cuda_stream) == s.cuda_stream


def test_read_probe_reads_every_byte(fc):
    """The probe's per-block sums of an all-ones buffer count its floats
    exactly (a ragged last block included)."""
    import torch
    n = 3 * 4096 + 904
    x = torch.ones(n, device="cuda")
    blocks = fc.fc_read_probe_blocks(4 * n)
    out = torch.full((blocks,), -1.0, device="cuda")
    fc.read_probe(x, out)
    torch.cuda.synchronize()
    assert out.cpu().tolist() == [4096.0, 4096.0, 4096.0, 904.0]


@pytest.mark.parametrize("order", ["tree", "linear"])
@pytest.mark.parametrize("dtype", ["f32", "f16"])
@pytest.mark.parametrize("K,max_blocks,vecs", [(1, 0, 1), (17, 0, 1), (100, 3, 1), (1024, 0, 1), (33, 1, 1),
                                               (1, 0, 2), (30, 2, 2), (128, 0, 2), (511, 1, 2)])
def test_resident_matches_oracle(fc, K, max_blocks, vecs, dtype, order):
    """The resident schedule (phase 1: reduce each block's tiles into LDS;
    phase 2: finish them from LDS), with tiles of 64 lanes x 1 vector
    (batches of 16) or x 2 vectors (batches of 4): reduce and steps with raw
    sum and broadcast (phase 3: one destination at a time, over one round or
    many), blocks with one tile or with many, both orders."""
    segs = table(14000 + K, dtype, nseg=5, max_len=3000 if K < 500 else 800)
    rng = np.random.default_rng(K + 3)
    opts = dict(schedule=3, max_blocks=max_blocks, vecs_per_thread=vecs)
    bad, _, _ = run_reduce(fc, segs, K, dtype, order, rng, opts=opts)
    assert bad == 0
    # signed zeros, subnormals, infinities and NaNs through the same loads and stack
    bad, _, _ = run_reduce(fc, segs, K, dtype, order, rng, opts=opts, special=True)
    assert bad == 0
    assert run_steps(fc, segs, K, dtype, order, rng, steps=2, opts=opts, with_out=True,
                     with_bcast=K <= 64) == 0


@pytest.mark.parametrize("schedule", [3, 4])
@pytest.mark.parametrize("dtype", ["f32", "f16"])
@pytest.mark.parametrize("K,max_blocks,vecs", [(5, 1, 1), (33, 2, 1), (130, 1, 1), (40, 1, 2)])
def test_resident_rounds_match_oracle(fc, K, max_blocks, vecs, dtype, schedule):
    """A plan larger than the grid's LDS takes several rounds (here with 1-3
    blocks of 160 tile slots each), one launch per round or all of them in
    one launch; every round's ranges are finished before the next round's
    reduce reuses the slots."""
    rows = [(0, 50000, 1, 1), (50048, 7, 2.0, 0.0), (50112, 60001, 1, 1), (110144, 200000, 1, 1)]
    p = fc.Plan(rows, K, dtype, "tree", schedule=schedule, max_blocks=max_blocks, vecs_per_thread=vecs)
    info = p.info()
    p.close()
    assert info.rounds >= 2 and info.grid == max_blocks and info.vecs_per_thread == vecs
    assert info.schedule == schedule
    rng = np.random.default_rng(K)
    opts = dict(schedule=schedule, max_blocks=max_blocks, vecs_per_thread=vecs)
    bad, _, _ = run_reduce(fc, rows, K, dtype, "tree", rng, opts=opts)
    assert bad == 0
    assert run_steps(fc, rows, K, dtype, "tree", rng, steps=2, opts=opts, with_out=True) == 0


def test_resident_plans_with_different_lds_interleave(fc):
    """Plans whose resident blocks need different amounts of LDS share the
    same kernel: creating a small plan after a large one must not break the
    large one's launches."""
    import torch
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    big_n = cus * 150 * 256  # 150 tiles per block
    K = 4
    rows_big = [(0, big_n, 1.0, 1.0)]
    rows_small = [(0, 3000, 1.0, 1.0)]
    rng = np.random.default_rng(77)
    big = fc.Plan(rows_big, K, "f32", "tree", schedule=3)
    small = fc.Plan(rows_small, K, "f32", "tree", schedule=3)
    # the small plan's 6 tiles of 512 take one round with or without
    # register-held tiles, so they sit in 6 LDS slots of 2 KiB
    assert big.info().lds_bytes == 160 * 1024 and small.info().lds_bytes == 6 * 2 * 1024
    reps = torch.from_numpy(rng.standard_normal((K, big_n), dtype=np.float32)).cuda()
    out = torch.full((big_n,), -1.0, device="cuda")
    big.tree_reduce(reps, out)
    small.tree_reduce(reps, out)
    big.tree_reduce(reps, out)
    torch.cuda.synchronize()
    x = reps.cpu().numpy()
    expect = (x[0] + x[1]) + (x[2] + x[3])
    assert same_bits(out.cpu().numpy(), expect) == 0
    big.close()
    small.close()


@pytest.mark.parametrize("batch", [1, 3, 1000, 65535])
def test_batch_not_a_power_of_two(fc, batch):
    """c = fl(1/batch) is inexact for most batches, so ga = s * c rounds: both
    sides compute c once on the host in fp32 and must agree bit for bit, in
    every schedule."""
    segs = table(15000 + batch, "f32", nseg=4, max_len=2500)
    for schedule in (1, 2, 3):
        rng = np.random.default_rng(batch + schedule)
        assert run_steps(fc, segs, 20, "f32", "tree", rng, steps=2, opts=dict(schedule=schedule),
                         batch=batch) == 0, schedule


@pytest.mark.parametrize("n,K,max_blocks,vecs,dtype", [
    (1000, 4, 0, 1, "f32"), (5_000_000, 8, 0, 1, "f32"), (40_000_000, 8, 0, 1, "f32"),
    (143_667_240, 16, 0, 1, "f32"), (143_667_240, 16, 0, 2, "f32"), (60_965_224, 128, 0, 2, "f32"),
    (60_965_224, 32, 0, 1, "f32"), (300_000, 8, 3, 1, "f32"), (300_000, 8, 3, 2, "f32"), (1, 1, 0, 1, "f32"),
    (60_965_224, 128, 0, 1, "f16"), (60_965_224, 600, 0, 1, "f16"), (5_000_000, 64, 0, 1, "f16"),
    (300_000, 16, 3, 1, "f16"), (1000, 4, 0, 1, "f16")])
def test_resident_partition(fc, n, K, max_blocks, vecs, dtype):
    """The resident plan's grid, rounds and LDS per block follow from the tile
    count, the CU's LDS and the tiles its waves hold in registers: rounds =
    ceil(tiles / (grid * (slots + 16 * rt))) for tiles of 64 * vecs vectors,
    each with 1 KiB * vecs of LDS (160 KiB per CU); rt = 4 register-held
    tiles per wave for fp32 tiles of 2 vectors with K < 32 and fp16 tiles of
    1 vector with K < 512 when they save rounds, else 0; a block's LDS holds
    the slots of as many tiles as it could be given in one round beyond its
    registers (a round's tiles, at most the CU's capacity), so that
    rebalanced ranges never need more."""
    import math
    import torch
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    p = fc.Plan([(0, n, 1, 1)], K, dtype, "tree", schedule=3, max_blocks=max_blocks, vecs_per_thread=vecs)
    info = p.info()
    p.close()
    tiles = (n // 4 + 64 * vecs - 1) // (64 * vecs) + (1 if n % 4 else 0)
    grid = min(cus, max_blocks) if max_blocks else cus
    grid = min(grid, tiles)
    slots = (160 * 1024) // (1024 * vecs)
    rt = (dtype == "f32" and vecs == 2 and K < 32) or (dtype == "f16" and vecs == 1 and K < 512)
    regs = 16 * 4 if rt else 0
    if regs and math.ceil(tiles / (grid * (slots + regs))) >= math.ceil(tiles / (grid * slots)):
        regs = 0
    rounds = max(1, math.ceil(tiles / (grid * (slots + regs))))
    per = max(1, min(slots + regs, max(1, math.ceil(tiles / rounds))) - regs)
    assert (info.ntiles, info.grid, info.rounds, info.lds_bytes) == (tiles, grid, rounds, per * 1024 * vecs), \
        (info.ntiles, info.grid, info.rounds, info.lds_bytes)
    assert info.lds_bytes <= 160 * 1024


@pytest.mark.parametrize("K,S", [(128, 16), (100, 16), (1024, 128), (37, 8)])
def test_sharded_reduction_equals_full_tree(fc, K, S):
    """The multi-GPU plan on one GPU: each of the runs of S aligned workers
    (one GPU's share) is reduced on its own, then the run sums are reduced in
    order by a plan over ceil(K / S) inputs -- the same bits as one plan over
    all K (the sharded allreduce design keeps parity)."""
    import torch
    n = 20000
    rng = np.random.default_rng(K + S)
    x = to_dev(rng.standard_normal((K, n), dtype=np.float32))
    rows = [(0, n, 1, 1)]
    full = torch.empty(n, device="cuda")
    p = fc.Plan(rows, K, "f32", "tree")
    p.tree_reduce(x, full)
    p.close()
    runs = [(i, min(S, K - i)) for i in range(0, K, S)]
    parts = torch.empty((len(runs), n), device="cuda")
    for r, (i, m) in enumerate(runs):
        q = fc.Plan(rows, m, "f32", "tree")
        q.tree_reduce([x[i + j] for j in range(m)], parts[r])
        q.close()
    top = torch.empty(n, device="cuda")
    q = fc.Plan(rows, len(runs), "f32", "tree")
    q.tree_reduce(parts, top)
    q.close()
    torch.cuda.synchronize()
    assert same_bits(top.cpu().numpy(), full.cpu().numpy()) == 0


@pytest.mark.parametrize("dtype", ["f32", "f16"])
@pytest.mark.parametrize("K,max_blocks,vecs,schedule", [(16, 8, 1, 3), (33, 16, 1, 3), (5, 1, 1, 3), (64, 3, 1, 3),
                                                        (40, 2, 2, 3), (5, 1, 1, 4), (40, 2, 2, 4)])
def test_balance_keeps_bits(fc, K, max_blocks, vecs, schedule, dtype):
    """fc_plan_balance after every step re-divides the resident tiles among
    the blocks by their XCDs' measured rates: every step before and after
    stays bit-exact with the oracle (update, raw sum, and for K <= 16 the
    broadcast copies), in one round over 8 or 16 blocks (every XCD) and in
    several rounds (1-3 blocks of 160 tile slots; one launch per round or
    all rounds in one launch, whose blocks add up their rounds' record); so
    does fc_broadcast on the rebalanced ranges."""
    segs = table(16000 + K, dtype, nseg=9)
    segs = segs + [(alloc_len(segs), 300000, 1.0, 1.0)]  # >= 32 tiles per block: launches record
    opts = dict(schedule=schedule, max_blocks=max_blocks, vecs_per_thread=vecs)
    p = fc.Plan(segs, K, dtype, "tree", **opts)
    info = p.info()
    assert p.balance() == [0.0] * 16  # nothing launched yet: no change, no rates
    p.close()
    assert info.grid == max_blocks
    if max_blocks <= 3:
        assert info.rounds >= 2
    rates = []
    bad = run_steps(fc, segs, K, dtype, "tree", np.random.default_rng(K), steps=4, opts=opts, with_out=True,
                    with_bcast=K <= 16, after_step=lambda plan: rates.append(plan.balance()))
    assert bad == 0
    ran = [r for r in rates[-1] if r > 0]
    assert 1 <= len(ran) <= min(8, info.grid)
    # fc_broadcast on rebalanced ranges
    import torch
    n = alloc_len(segs)
    src = host_replicas(np.random.default_rng(K + 1), 1, n, np.float32, special=True)[0]
    p = fc.Plan(segs, K, dtype, "tree", **opts)
    reps = to_dev(host_replicas(np.random.default_rng(K + 2), K, n, np.float16 if dtype == "f16" else np.float32))
    w_d, v_d = torch.zeros(n, device="cuda"), torch.zeros(n, device="cuda")
    p.step(reps, w_d, v_d, LR, MU, WD, 256)
    p.balance()
    kb = K
    dst = torch.full((K, n), -2.0, device="cuda")
    p.broadcast(to_dev(src), dst)
    torch.cuda.synchronize()
    got = dst[:kb].cpu().numpy()
    p.close()
    expect = oracle.broadcast(segs, src, [np.full(n, -2.0, np.float32) for _ in range(kb)])
    assert sum(same_bits(got[k], expect[k]) for k in range(kb)) == 0


def test_balance_full_grid_reduce(fc):
    """One round over the whole grid (every XCD): the raw sums before and
    after rebalancing are the same bits, equal to the pairwise tree of 4."""
    import torch
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    n = cus * 120 * 256 + 13
    K = 4
    rng = np.random.default_rng(5)
    x = rng.standard_normal((K, n + 3), dtype=np.float32)
    reps = to_dev(x)
    plan = fc.Plan([(0, n, 1.0, 1.0)], K, "f32", "tree", schedule=3)
    assert plan.info().rounds == 1 and plan.info().grid == cus
    out = torch.full((n + 3,), -1.0, device="cuda")
    plan.tree_reduce(reps, out)
    rates = plan.balance()
    assert sum(1 for r in rates if r > 0) == min(8, cus)
    first = out.cpu().numpy()
    out.fill_(-1.0)
    for _ in range(3):
        plan.tree_reduce(reps, out)
        plan.balance()
    torch.cuda.synchronize()
    expect = (x[0] + x[1]) + (x[2] + x[3])
    expect[n:] = -1.0
    assert same_bits(first, expect) == 0
    assert same_bits(out.cpu().numpy(), expect) == 0
    plan.close()


def test_balance_leaves_other_schedules_and_small_plans(fc):
    """Fused plans, and resident plans whose blocks take fewer than 32 tiles
    per round (here one tile per block), record nothing and keep their
    shares: fc_plan_balance returns no rates."""
    segs = table(17000, "f32", nseg=4)
    rng = np.random.default_rng(3)
    n = alloc_len(segs)
    reps = to_dev(host_replicas(rng, 8, n, np.float32))
    w, v = to_dev(np.zeros(n, np.float32)), to_dev(np.zeros(n, np.float32))
    for sched in (1, 3):
        p = fc.Plan(segs, 8, "f32", "tree", schedule=sched)
        p.step(reps, w, v, LR, MU, WD, 256)
        assert p.balance() == [0.0] * 16, sched
        p.close()


def test_graph_replays_after_balance(fc):
    """A graph captured before fc_plan_balance replays with the new shares
    (the range table changes in place; the launches' LDS already covers any
    share), bit-identical to an eager twin plan."""
    import torch
    segs = table(18000, "f32", nseg=9)  # 110 tiles, 55 per block of 2: launches record
    K = 24
    n = alloc_len(segs)
    rng = np.random.default_rng(11)
    reps = to_dev(host_replicas(rng, K, n, np.float32, scale=0.01))
    w0 = rng.standard_normal(n, dtype=np.float32) * np.float32(0.05)
    wa, va = to_dev(w0), torch.zeros(n, device="cuda")
    wb, vb = to_dev(w0), torch.zeros(n, device="cuda")
    pa = fc.Plan(segs, K, "f32", "tree", schedule=3, max_blocks=2)
    pb = fc.Plan(segs, K, "f32", "tree", schedule=3, max_blocks=2)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        pa.step(reps, wa, va, LR, MU, WD, 256)
    s.synchronize()
    pb.step(reps, wb, vb, LR, MU, WD, 256)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        pa.step(reps, wa, va, LR, MU, WD, 256)
    for _ in range(3):
        g.replay()
        torch.cuda.synchronize()
        assert sum(1 for r in pa.balance(stream=s) if r > 0) == 2
        pb.step(reps, wb, vb, LR, MU, WD, 256)
        torch.cuda.synchronize()
        assert same_bits(wa.cpu().numpy(), wb.cpu().numpy()) == 0
        assert same_bits(va.cpu().numpy(), vb.cpu().numpy()) == 0
    pa.close()
    pb.close()


def test_graph_replays_broadcast(fc):
    """fc_step with the broadcast and fc_broadcast captured in one HIP graph
    on a resident plan of several rounds: every replay (eager work and a
    synchronization between replays, the source changed eagerly each time)
    gives every destination the oracle's copy of the source and of w'."""
    import torch
    segs = table(19000, "f32", nseg=6, max_len=20000)
    segs = segs + [(alloc_len(segs), 100000, 1.0, 1.0)]  # > 144 tiles of 512: several rounds
    K = 5
    n = alloc_len(segs)
    rng = np.random.default_rng(13)
    reps = to_dev(host_replicas(rng, K, n, np.float32, scale=0.01))
    w = to_dev(rng.standard_normal(n, dtype=np.float32) * np.float32(0.05))
    v = torch.zeros(n, device="cuda")
    src = torch.zeros(n, device="cuda")
    d1 = torch.full((K, n), -2.0, device="cuda")
    d2 = torch.full((K, n), -3.0, device="cuda")
    # one plan per set of destination pointers: a captured call keeps its
    # plan's pointer tables
    plan = fc.Plan(segs, K, "f32", "tree", schedule=3, max_blocks=1)
    pb = fc.Plan(segs, K, "f32", "tree", schedule=3, max_blocks=1)
    assert plan.info().rounds > 1
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        plan.step(reps, w, v, LR, MU, WD, 256, bcast=d1)
        pb.broadcast(src, d2)
    s.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        plan.step(reps, w, v, LR, MU, WD, 256, bcast=d1)
        pb.broadcast(src, d2)
    w_h, v_h = w.cpu().numpy(), v.cpu().numpy()
    for i in range(3):
        x = host_replicas(np.random.default_rng(100 + i), 1, n, np.float32, special=True)[0]
        src.copy_(to_dev(x))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        w_h, v_h, _, _ = oracle.step(segs, list(reps.cpu().numpy()), w_h, v_h, LR, MU, WD, 256)
        assert same_bits(w.cpu().numpy(), w_h) == 0 and same_bits(v.cpu().numpy(), v_h) == 0
        want1 = oracle.broadcast(segs, w_h, [np.full(n, -2.0, np.float32) for _ in range(K)])
        want2 = oracle.broadcast(segs, x, [np.full(n, -3.0, np.float32) for _ in range(K)])
        got1, got2 = d1.cpu().numpy(), d2.cpu().numpy()
        assert sum(same_bits(got1[k], want1[k]) for k in range(K)) == 0, i
        assert sum(same_bits(got2[k], want2[k]) for k in range(K)) == 0, i
    plan.close()
    pb.close()


def test_capture_refuses_a_table_change(fc):
    """Inside a graph capture a call whose pointers differ from the plan's
    previous call, or a call with per-kernel timing on, returns FC_EINVAL
    and enqueues nothing; the capture's other calls still replay
    correctly."""
    import torch
    segs = table(20000, "f32", nseg=3, max_len=3000)
    K = 3
    n = alloc_len(segs)
    rng = np.random.default_rng(17)
    ra = to_dev(host_replicas(rng, K, n, np.float32))
    rb = ra.clone()
    out = torch.full((n,), -1.0, device="cuda")
    plan = fc.Plan(segs, K, "f32", "tree")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        plan.tree_reduce(ra, out)
    s.synchronize()
    g = torch.cuda.CUDAGraph()
    codes = []
    rows_a = [int(x) for x in fc._rows(ra)]
    with torch.cuda.graph(g, stream=s):
        plan.tree_reduce(ra, out)
        codes.append(fc.fc_tree_reduce(plan.handle, [int(x) for x in fc._rows(rb)], out.data_ptr(),
                                       s.cuda_stream))
        # per-kernel timing is refused under capture too
        plan.set_timing(True)
        codes.append(fc.fc_tree_reduce(plan.handle, rows_a, out.data_ptr(), s.cuda_stream))
        plan.set_timing(False)
    assert codes == [fc._fc.FC_EINVAL, fc._fc.FC_EINVAL]
    assert all(n == 0 for n, _ in plan.read_timing().values())
    out.fill_(-1.0)
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    expect = oracle.tree_reduce(segs, list(ra.cpu().numpy()), out=np.full(n, -1.0, np.float32))
    assert same_bits(out.cpu().numpy(), expect) == 0
    plan.close()


def test_balance_refused_under_capture(fc):
    """fc_plan_balance would wait on the stream: while that stream is being
    captured it returns FC_EINVAL without waiting, the capture stays valid
    and its step replays bit-exact with an eager twin plan."""
    import torch
    segs = table(18000, "f32", nseg=9)  # 110 tiles, 55 per block of 2: launches record
    K = 24
    n = alloc_len(segs)
    rng = np.random.default_rng(19)
    reps = to_dev(host_replicas(rng, K, n, np.float32, scale=0.01))
    w0 = rng.standard_normal(n, dtype=np.float32) * np.float32(0.05)
    wa, va = to_dev(w0), torch.zeros(n, device="cuda")
    wb, vb = to_dev(w0), torch.zeros(n, device="cuda")
    pa = fc.Plan(segs, K, "f32", "tree", schedule=3, max_blocks=2)
    pb = fc.Plan(segs, K, "f32", "tree", schedule=3, max_blocks=2)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        pa.step(reps, wa, va, LR, MU, WD, 256)
    s.synchronize()
    pb.step(reps, wb, vb, LR, MU, WD, 256)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        pa.step(reps, wa, va, LR, MU, WD, 256)
        rc, _ = fc.fc_plan_balance(pa.handle, s.cuda_stream)
    assert rc == fc._fc.FC_EINVAL
    g.replay()
    pb.step(reps, wb, vb, LR, MU, WD, 256)
    torch.cuda.synchronize()
    assert same_bits(wa.cpu().numpy(), wb.cpu().numpy()) == 0
    assert same_bits(va.cpu().numpy(), vb.cpu().numpy()) == 0
    pa.close()
    pb.close()


def test_balance_drains_the_plans_stream(fc):
    """Steps on a side stream, fc_plan_balance called with the null stream:
    the call drains the stream the plan last ran on before it replaces the
    range table, and every later step stays bit-exact."""
    import torch
    segs = table(19000, "f32", nseg=9)
    K = 20
    n = alloc_len(segs)
    rng = np.random.default_rng(12)
    reps_h = host_replicas(rng, K, n, np.float32, scale=0.01)
    w = rng.standard_normal(n, dtype=np.float32) * np.float32(0.05)
    v = np.zeros(n, np.float32)
    p = fc.Plan(segs, K, "f32", "tree", schedule=3, max_blocks=2)  # 106 tiles: 53 per block, launches record
    reps, w_d, v_d = to_dev(reps_h), to_dev(w), to_dev(v)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    for i in range(4):
        with torch.cuda.stream(side):
            p.step(reps, w_d, v_d, LR, MU, WD, 256)
        w, v, _, _ = oracle.step(segs, list(reps_h), w, v, LR, MU, WD, 256)
        rates = p.balance(stream=0)
        assert any(r > 0 for r in rates)
    side.synchronize()
    assert same_bits(w_d.cpu().numpy(), w) == 0 and same_bits(v_d.cpu().numpy(), v) == 0
    p.close()


@pytest.mark.parametrize("K,vecs,per_block,dtype", [(40, 1, 160, "f32"), (6, 2, 144, "f32"), (40, 1, 224, "f16")])
def test_balance_with_full_lds_keeps_equal_shares(fc, K, vecs, per_block, dtype):
    """Two blocks whose equal share of each round already fills the block
    (2 rounds: 160 LDS slots of 256-element tiles; with fp32 tiles of 2
    vectors, 80 slots and 64 tiles of 512 elements in its waves' registers;
    with fp16 replicas, 160 slots and 64 tiles in registers): no unequal
    division fits, so the shares fc_plan_balance writes stay equal; the steps
    after it stay bit-exact."""
    n = 2 * 2 * per_block * 256 * vecs
    segs = [(0, n, 1.0, 1.0)]
    opts = dict(schedule=3, max_blocks=2, vecs_per_thread=vecs)
    p = fc.Plan(segs, K, dtype, "tree", **opts)
    info = p.info()
    p.close()
    assert (info.ntiles, info.rounds, info.lds_bytes) == (4 * per_block, 2, 160 * 1024)
    rates = []
    bad = run_steps(fc, segs, K, dtype, "tree", np.random.default_rng(21), steps=3, opts=opts,
                    after_step=lambda plan: rates.append(plan.balance()))
    assert bad == 0
    assert sum(1 for r in rates[-1] if r > 0) == 2


@pytest.mark.parametrize("K,dtype,vecs", [(1, "f32", 2), (3, "f32", 2), (16, "f32", 2), (31, "f32", 2),
                                          (16, "f32", 1), (16, "f16", 1), (128, "f16", 1), (300, "f16", 1),
                                          (600, "f16", 1)])
@pytest.mark.parametrize("order", ["tree", "linear"])
def test_resident_register_and_lds_tiles(fc, K, dtype, vecs, order):
    """fp32 plans with tiles of 2 vectors (512 elements) and K < 32, and fp16
    plans (tiles of 256 elements) with K < 512, keep each wave's first 4
    tiles of a round in registers and the rest in LDS when that saves
    rounds: here with one block, and with two for most cases, every round
    uses both (the other shapes, LDS only, over many rounds); reduce, steps
    with raw sum and broadcast, and fc_broadcast (which stages a block's
    range through its LDS slots in pieces) against the oracle; ragged
    segments and tail tiles."""
    import math
    import torch
    rng = np.random.default_rng(K * 3 + vecs + (order == "tree") + (dtype == "f16") * 7)
    big = (300_000 if dtype == "f16" else 230_000) if K < 200 else 120_000
    segs = table(21000 + K, dtype, nseg=7, max_len=4000) + [(0, big, 1.0, 1.0), (0, 1001, 2.0, 0.0)]
    off = 0
    rows = []
    for _, m, lm, dm in segs:  # re-laid end to end, 64-element aligned, so the big segment sits mid-table
        rows.append((off, m, lm, dm))
        off = (off + m + 63) // 64 * 64
    for max_blocks in (1, 2):
        opts = dict(schedule=3, max_blocks=max_blocks, vecs_per_thread=vecs)
        p = fc.Plan(rows, K, dtype, order, **opts)
        info = p.info()
        slots = 160 // vecs
        rt = (dtype == "f32" and vecs == 2 and K < 32) or (dtype == "f16" and K < 512)
        lds_rounds = math.ceil(info.ntiles / (max_blocks * slots))
        rt_rounds = math.ceil(info.ntiles / (max_blocks * (slots + 64)))
        used = rt and rt_rounds < lds_rounds
        assert info.rounds == (rt_rounds if used else lds_rounds) >= 1, (info.ntiles, info.rounds)
        assert used or not rt or max_blocks == 2, (info.ntiles, info.rounds)
        assert info.ntiles > max_blocks * (64 if used else 0), info.ntiles
        p.close()
        bad, _, _ = run_reduce(fc, rows, K, dtype, order, rng, opts=opts)
        assert bad == 0, max_blocks
        assert run_steps(fc, rows, K, dtype, order, rng, steps=2, opts=opts, with_out=True,
                         with_bcast=K <= 3) == 0, max_blocks
    n = alloc_len(rows)
    src = host_replicas(rng, 1, n, np.float32, special=True)[0]
    expect = oracle.broadcast(rows, src, [np.full(n, -2.0, np.float32) for _ in range(K)])
    p = fc.Plan(rows, K, dtype, order, schedule=3, max_blocks=1, vecs_per_thread=vecs)
    dst = torch.full((K, n), -2.0, device="cuda")
    p.broadcast(to_dev(src), dst)
    torch.cuda.synchronize()
    p.close()
    got = dst.cpu().numpy()
    assert sum(same_bits(got[k], expect[k]) for k in range(K)) == 0


@pytest.mark.parametrize("schedule", [2, 3])
def test_calls_on_several_streams_are_ordered(fc, schedule):
    """Steps of one plan on three streams, each on its own w, v, with the
    replica table replaced between them: every call runs after the plan's
    previous call whatever its stream, so a table replaced for a later call
    is never read by an earlier one still running, and the two-pass raw-sum
    scratch never serves two calls at once.  Every result equals the
    oracle's, applied in the order of the calls."""
    import torch
    K = 70
    segs = [(0, 1 << 21, 1.0, 1.0), ((1 << 21) + 64, 1000, 1.0, 1.0)]
    n = alloc_len(segs)
    rng = np.random.default_rng(77)
    sets_h = [host_replicas(rng, K, n, np.float32, scale=0.01) for _ in range(2)]
    sets = [to_dev(r) for r in sets_h]
    ws_h = [rng.standard_normal(n, dtype=np.float32) * np.float32(0.05) for _ in range(4)]
    vs_h = [np.zeros(n, np.float32) for _ in range(4)]
    ws, vs = [to_dev(w) for w in ws_h], [to_dev(v) for v in vs_h]
    p = fc.Plan(segs, K, "f32", "tree", schedule=schedule)
    streams = [torch.cuda.Stream() for _ in range(3)]
    for st in streams:
        st.wait_stream(torch.cuda.current_stream())
    # (stream, replica set, w/v set)
    calls = [(0, 0, 0), (1, 0, 1), (2, 1, 2), (0, 0, 3), (1, 1, 0), (2, 1, 1), (0, 0, 2)]
    for si, r, j in calls:
        with torch.cuda.stream(streams[si]):
            p.step(sets[r], ws[j], vs[j], LR, MU, WD, 256)
        ws_h[j], vs_h[j], _, _ = oracle.step(segs, list(sets_h[r]), ws_h[j], vs_h[j], LR, MU, WD, 256)
    torch.cuda.synchronize()
    p.close()
    for j in range(4):
        assert same_bits(ws[j].cpu().numpy(), ws_h[j]) == 0, j
        assert same_bits(vs[j].cpu().numpy(), vs_h[j]) == 0, j

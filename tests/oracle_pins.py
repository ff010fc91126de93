"""Pins for the oracle: facts fixed by the paper and by the mathematics, not by
the oracle itself.  Each pin raises AssertionError when it does not hold.

Collected by test_oracle_pins.py against the real oracle and, with planted
mistakes, against mutated copies of it (each mutant must fail some pin).
"""
import math
import os

import numpy as np

import oracle

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
U = 2.0 ** -24  # unit roundoff of binary32


def _bits(a):
    return np.asarray(a, dtype=np.float32).view(np.uint32)


def _same(a, b):
    """Bitwise equality, except that any NaN equals any NaN."""
    a = np.asarray(a, dtype=np.float32)
    b = np.asarray(b, dtype=np.float32)
    nan = np.isnan(a) & np.isnan(b)
    return bool(np.all(nan | (_bits(a) == _bits(b))))


def _reduce(x, order="tree"):
    """Reduce a (K, n) array over its segment [0, n) with the oracle."""
    K, n = x.shape
    return oracle.tree_reduce([(0, n)], list(x), order=order)


# ------------------------------------------------------------------ widening
def pin_f16_widen_exhaustive():
    """All 65536 binary16 patterns widen exactly as numpy's float16->float32
    conversion does (a library routine), both through the scalar entry and
    through a K=1 reduction of fp16 replicas."""
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    ref = bits.view(np.float16).astype(np.float32)
    assert _same(oracle.f16_to_f32(bits), ref)
    out = _reduce(bits.view(np.float16)[None, :])
    assert _same(out, ref)


# ------------------------------------------------------------------ tree sum
def pin_k1_identity():
    """With one worker the aggregate is that worker's vector, bit for bit,
    special values included."""
    special = np.array([0x00000000, 0x80000000, 0x00000001, 0x807fffff, 0x00800000, 0x7f7fffff,
                        0x7f800000, 0xff800000, 0x7fc00000, 0x3f800000, 0xbf800001],
                       dtype=np.uint32).view(np.float32)
    rng = np.random.default_rng(1)
    x = np.concatenate([special, rng.standard_normal(500).astype(np.float32)])[None, :]
    for order in ("tree", "linear"):
        assert _same(_reduce(x, order), x[0])


def pin_all_ones():
    """K copies of 1.0 sum to exactly K in either order (all partial sums are
    small integers)."""
    for K in list(range(1, 131)) + [255, 256, 1000, 1024]:
        x = np.ones((K, 3), dtype=np.float32)
        for order in ("tree", "linear"):
            assert np.all(_reduce(x, order) == np.float32(K)), (K, order)


def pin_integer_exact():
    """Integer-valued inputs whose partial sums stay below 2^24 in magnitude
    are added exactly, so the result is the integer sum and does not depend
    on the order (fp32 and fp16 storage)."""
    rng = np.random.default_rng(2)
    for K in (2, 3, 5, 7, 8, 13, 32, 100, 128):
        xi = rng.integers(-(1 << 16), 1 << 16, size=(K, 257))
        exact = xi.sum(axis=0)
        x = xi.astype(np.float32)
        t, lin = _reduce(x, "tree"), _reduce(x, "linear")
        assert np.array_equal(t.astype(np.int64), exact)
        assert _same(t, lin)
        xh = rng.integers(-2048, 2049, size=(K, 129))
        t16 = _reduce(xh.astype(np.float16), "tree")
        assert np.array_equal(t16.astype(np.int64), xh.sum(axis=0))


def pin_fsum_bound():
    """Against the exactly rounded sum (math.fsum), the error is within the
    pairwise-summation bound gamma_d * sum|x| with d = ceil(log2 K) for the
    binary tree, d = K-1 for the linear order (Higham, Accuracy and Stability
    of Numerical Algorithms, Sec. 4.2)."""
    rng = np.random.default_rng(3)
    for K in (2, 3, 5, 7, 8, 16, 31, 32, 64, 100, 128):
        x = (rng.standard_normal((K, 300)) * 10.0 ** rng.integers(-3, 3, size=(K, 1))).astype(np.float32)
        for order, d in (("tree", math.ceil(math.log2(K))), ("linear", K - 1)):
            got = _reduce(x, order).astype(np.float64)
            gam = d * U / (1 - d * U)
            for i in range(x.shape[1]):
                col = x[:, i].astype(np.float64)
                exact = math.fsum(col)
                assert abs(got[i] - exact) <= gam * np.abs(col).sum() * (1 + 1e-12), (K, order, i)


def _golden_rows(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(line.split())
    return rows


def pin_order_golden():
    """Hand-worked examples in which tree and linear order give different
    bits (tests/golden/order_example.txt)."""
    for row in _golden_rows("order_example.txt"):
        vals = np.array([int(h, 16) for h in row], dtype=np.uint32)
        x = vals[:-2].view(np.float32)
        tree_bits, lin_bits = int(vals[-2]), int(vals[-1])
        xs = np.repeat(x[:, None], 2, axis=1)
        assert int(_bits(_reduce(xs, "tree"))[0]) == tree_bits
        assert int(_bits(_reduce(xs, "linear"))[0]) == lin_bits


def _balanced(x):
    """Fig. 3b for K a power of two: the sum of a subtree is the sum of its
    left half plus the sum of its right half (each add one fp32 rounding)."""
    K = x.shape[0]
    if K == 1:
        return x[0]
    return _balanced(x[:K // 2]) + _balanced(x[K // 2:])


def _binomial_blocks(x):
    """Same tree for any K, stated another way: split the K leaves into
    consecutive blocks whose sizes are the powers of two in K's binary
    representation, largest first; sum each block as a balanced tree; then
    add the block sums from the smallest block upwards, each new block on the
    left."""
    K = x.shape[0]
    sizes = [1 << b for b in range(K.bit_length() - 1, -1, -1) if K >> b & 1]
    blocks, start = [], 0
    for s in sizes:
        blocks.append(_balanced(x[start:start + s]))
        start += s
    acc = blocks[-1]
    for b in reversed(blocks[:-1]):
        acc = b + acc
    return acc


def pin_tree_structure():
    """The oracle's level-by-level pairing equals the balanced tree for K a
    power of two and the block decomposition for every K up to 130."""
    rng = np.random.default_rng(4)
    for K in range(1, 131):
        x = (rng.standard_normal((K, 64)) * np.exp(rng.standard_normal((K, 1)) * 3)).astype(np.float32)
        got = _reduce(x, "tree")
        assert _same(got, _binomial_blocks(x)), K
        if K & (K - 1) == 0:
            assert _same(got, _balanced(x)), K


def pin_tree_shards():
    """Sharding over workers keeps the tree's bits (Sec. 6.2 tree over p
    nodes): cut the K leaves into aligned runs of S = 2^m (the last one
    shorter), reduce each run, then reduce the run sums in order -- the result
    is the tree over all K leaves.  This is what lets G GPUs each reduce their
    own workers' subtree and one owner combine the G partials."""
    rng = np.random.default_rng(6)
    for K, S in ((128, 16), (128, 1), (128, 128), (100, 16), (37, 8), (1000, 64), (7, 4), (130, 32)):
        x = (rng.standard_normal((K, 48)) * np.exp(rng.standard_normal((K, 1)) * 3)).astype(np.float32)
        parts = np.stack([_reduce(x[i:i + S], "tree") for i in range(0, K, S)])
        assert _same(_reduce(parts, "tree"), _reduce(x, "tree")), (K, S)


def pin_linear_structure():
    """Parameter-server order: the running sum x0+x1, then +x2, ... (numpy
    cumulative sum in float32 adds left to right)."""
    rng = np.random.default_rng(5)
    for K in (1, 2, 3, 9, 64, 128):
        x = rng.standard_normal((K, 77)).astype(np.float32)
        acc = x[0].copy()
        for k in range(1, K):
            acc = acc + x[k]
        assert _same(_reduce(x, "linear"), acc)
        assert _same(_reduce(x, "linear"), np.cumsum(x, axis=0, dtype=np.float32)[-1])


def pin_ieee_special_sums():
    """IEEE facts: +inf + -inf is NaN; inf absorbs finite values; +0 + -0 is
    +0 and -0 + -0 is -0 under round-to-nearest."""
    inf, nz = np.float32(np.inf), np.float32(-0.0)
    x = np.array([[1, inf, inf, 0.0, nz], [2, -inf, 1, nz, nz], [3, 5, 1, 0.0, nz], [4, 7, 1, nz, nz]],
                 dtype=np.float32)
    for order in ("tree", "linear"):
        r = _reduce(x, order)
        assert r[0] == 10 and np.isnan(r[1]) and r[2] == inf
        assert _bits(r)[3] == 0 and _bits(r)[4] == 0x80000000


def pin_ragged_segments_and_padding():
    """Only segment elements are written; every gap keeps its old value; each
    segment element equals the reduction of that element alone."""
    rng = np.random.default_rng(6)
    segs = [(0, 5), (8, 1), (12, 17), (40, 3)]
    K = 6
    x = rng.standard_normal((K, 48)).astype(np.float32)
    out = np.full(48, 123.25, dtype=np.float32)
    oracle.tree_reduce(segs, list(x), out=out)
    inside = np.zeros(48, bool)
    for o, n in segs:
        inside[o:o + n] = True
    assert np.all(out[~inside] == np.float32(123.25))
    for i in np.flatnonzero(inside):
        single = oracle.tree_reduce([(0, 1)], [x[k, i:i + 1] for k in range(K)])
        assert _same(out[i], single[0])


# ------------------------------------------------------------------ SGD
def pin_sgd_golden():
    """Hand-worked steps with exact dyadic values (tests/golden/sgd_example.txt),
    and with per-segment multipliers (tests/golden/sgd_multipliers_example.txt)."""
    for row in _golden_rows("sgd_example.txt"):
        s, batch, lr, mu, wd, w, v, w1, v1 = [float(t) for t in row]
        wn, vn = oracle.sgd_step([(0, 1)], np.float32([w]), np.float32([v]), np.float32([s]),
                                 lr, mu, wd, int(batch))
        assert wn[0] == np.float32(w1) and vn[0] == np.float32(v1), row
    for row in _golden_rows("sgd_multipliers_example.txt"):
        s, batch, lr, mu, wd, lm, dm, w, v, w1, v1 = [float(t) for t in row]
        wn, vn = oracle.sgd_step([(0, 1, lm, dm)], np.float32([w]), np.float32([v]), np.float32([s]),
                                 lr, mu, wd, int(batch))
        assert wn[0] == np.float32(w1) and vn[0] == np.float32(v1), row


def _sgd_inputs(rng, n):
    # magnitudes chosen so that every term of the update matters
    s = (rng.standard_normal(n) * 2.5).astype(np.float32)
    w = (rng.standard_normal(n) * 0.2).astype(np.float32)
    v = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    return s, w, v


def pin_sgd_fp64_bound():
    """The update evaluated in fp64 from the same fp32 inputs agrees within
    the forward error bound of the six fp32 operations:
      |dv'| <= 4u (|mu v| + |lr_j| (|ga| + |wd_j w|)),
      |dw'| <= u |w - v'| + (1+u) |dv'|,
    with per-segment lr/decay multipliers and a power-of-two batch (so 1/batch
    is exact)."""
    rng = np.random.default_rng(7)
    segs = [(0, 300, 1.0, 1.0), (300, 200, 2.0, 0.0), (512, 100, 0.5, 3.0)]
    n = 612
    s, w, v = _sgd_inputs(rng, n)
    lr, mu, wd, batch = 0.1, 0.9, 0.05, 256
    wn, vn = oracle.sgd_step(segs, w, v, s, lr, mu, wd, batch)
    for off, ln, lm, dm in segs:
        sl = slice(off, off + ln)
        lr_j = float(np.float32(lr) * np.float32(lm))
        wd_j = float(np.float32(wd) * np.float32(dm))
        ga = s[sl].astype(np.float64) / batch
        dec = wd_j * w[sl].astype(np.float64)
        mom = float(np.float32(mu)) * v[sl].astype(np.float64)
        v64 = mom + lr_j * (ga + dec)
        w64 = w[sl].astype(np.float64) - v64
        bv = 4 * U * (np.abs(mom) + abs(lr_j) * (np.abs(ga) + np.abs(dec))) * 1.001
        bw = U * np.abs(w64) + (1 + U) * bv * 1.001
        assert np.all(np.abs(vn[sl] - v64) <= bv), (off, lm, dm)
        assert np.all(np.abs(wn[sl] - w64) <= bw), (off, lm, dm)


def pin_sgd_closed_forms():
    """Special cases with closed forms:
      lr = 0                    -> v' = mu*v exactly, w' = w - mu*v (one rounding)
      mu = wd = 0, v = 0, lr = 1 -> v' = s * 2^-e exactly (batch = 2^e), the
                                   average of Sec. 6; w' = w - v'
      s = 0, wd = 0             -> v' = mu*v: velocity decays geometrically
    """
    rng = np.random.default_rng(8)
    s, w, v = _sgd_inputs(rng, 256)
    seg = [(0, 256)]
    wn, vn = oracle.sgd_step(seg, w, v, s, 0.0, 0.9, 5e-4, 256)
    mv = np.float32(0.9) * v
    assert np.all(vn == mv) and np.all(wn == w - mv)
    for e in (0, 5, 8, 10):
        wn, vn = oracle.sgd_step(seg, w, np.zeros_like(v), s, 1.0, 0.0, 0.0, 1 << e)
        assert _same(vn, np.ldexp(s, -e).astype(np.float32))
        assert np.all(wn == w - vn)
    vv = v.copy()
    for _ in range(3):
        _, vv2 = oracle.sgd_step(seg, w, vv, np.zeros_like(s), 0.01, 0.5, 0.0, 256)
        assert np.all(vv2 == np.ldexp(vv, -1).astype(np.float32))
        vv = vv2


def pin_broadcast():
    """Every worker receives the same bits over the segments; gaps untouched."""
    rng = np.random.default_rng(9)
    src = rng.standard_normal(40).astype(np.float32)
    dsts = [np.full(40, -7.0, dtype=np.float32) for _ in range(5)]
    oracle.broadcast([(0, 9), (16, 20)], src, dsts)
    for d in dsts:
        assert _same(d[:9], src[:9]) and _same(d[16:36], src[16:36])
        assert np.all(d[9:16] == -7.0) and np.all(d[36:] == -7.0)


def pin_step_composition():
    """The whole step is reduce, then SGD on the raw sum, then broadcast of w'
    (Fig. 3: sum up the tree, send back down, workers apply the update)."""
    rng = np.random.default_rng(10)
    segs = [(0, 33, 1.0, 1.0), (64, 40, 2.0, 0.0)]
    K = 5
    x = rng.standard_normal((K, 104)).astype(np.float32)
    w = rng.standard_normal(104).astype(np.float32)
    v = rng.standard_normal(104).astype(np.float32) * np.float32(1e-3)
    out = np.zeros(104, np.float32)
    dst = [np.zeros(104, np.float32) for _ in range(K)]
    w1, v1, _, _ = oracle.step(segs, list(x), w, v, 0.01, 0.9, 5e-4, 256, out=out, bcast=dst)
    g = oracle.tree_reduce(segs, list(x))
    w2, v2 = oracle.sgd_step(segs, w, v, g, 0.01, 0.9, 5e-4, 256)
    assert _same(out, g) and _same(w1, w2) and _same(v1, v2)
    for d in dst:
        assert _same(d[:33], w1[:33]) and _same(d[64:104], w1[64:104])


# ------------------------------------------------------------------ learning-rate policies
def pin_lr_paper_values():
    """Sec. 7.2: NiN at batch 256 starts at 0.01 and is divided by 10 twice;
    at batch 1024 the rate is scaled by the same factor as the batch (0.04,
    Table 2).  Sec. 7.3: GoogLeNet at batch 1024 starts at 0.08."""
    step = dict(kind="step", base_lr=0.01, gamma=0.1, stepsize=1000)
    assert oracle.lr_at(iter=0, batch=256, **step) == np.float32(0.01)
    assert oracle.lr_at(iter=999, batch=256, **step) == np.float32(0.01)
    assert oracle.lr_at(iter=1000, batch=256, **step) == np.float32(0.001)
    assert oracle.lr_at(iter=2000, batch=256, **step) == np.float32(0.0001)
    assert oracle.lr_at("fixed", 0, 1024, 0.01, base_batch=256) == np.float32(0.04)
    assert oracle.lr_at("fixed", 0, 256, 0.01, base_batch=256) == np.float32(0.01)
    assert oracle.lr_at("poly", 0, 1024, 0.08, max_iter=10, power=0.5) == np.float32(0.08)


def pin_lr_poly_closed_forms():
    """Sec. 7.3 poly policy base * (1 - iter/max_iter)^power: the end of the
    run is 0; power 1 is a straight line; power 0.5 and 2 at points where the
    root and square are exact."""
    assert oracle.lr_at("poly", 8, 32, 0.5, max_iter=8, power=0.5) == 0.0
    assert oracle.lr_at("poly", 3, 32, 0.5, max_iter=8, power=1.0) == np.float32(0.3125)
    assert oracle.lr_at("poly", 3, 32, 0.08, max_iter=4, power=0.5) == np.float32(0.04)
    assert oracle.lr_at("poly", 1, 32, 0.08, max_iter=2, power=2.0) == np.float32(0.02)
    for bad in (dict(kind="poly", iter=9, max_iter=8), dict(kind="step", iter=1, stepsize=0),
                dict(kind="fixed", iter=-1)):
        kw = dict(batch=32, base_lr=0.1)
        kw.update(bad)
        try:
            oracle.lr_at(**kw)
        except ValueError:
            continue
        raise AssertionError(f"invalid policy accepted: {bad}")


PINS = [pin_f16_widen_exhaustive, pin_k1_identity, pin_all_ones, pin_integer_exact, pin_fsum_bound,
        pin_order_golden, pin_tree_structure, pin_tree_shards, pin_linear_structure, pin_ieee_special_sums,
        pin_ragged_segments_and_padding, pin_sgd_golden, pin_sgd_fp64_bound, pin_sgd_closed_forms,
        pin_broadcast, pin_step_composition, pin_lr_paper_values, pin_lr_poly_closed_forms]

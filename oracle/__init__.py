"""Oracle for the FireCaffe gradient aggregation + SGD step (numpy front end).

TEST INFRASTRUCTURE ONLY.  The arithmetic lives in ``fc_oracle.c`` (scalar C,
``-ffp-contract=off``); this module only marshals numpy arrays into it with
ctypes.  Only the tests, the smoke check and the benchmark's CPU-baseline leg
may import it; the HIP library never does, and this module imports nothing
from the HIP package.

Functions follow the paper's problem statement (Sec. 6 "Implementing efficient
data parallel training", Sec. 6.1 "Parameter server", Sec. 6.2 "Reduction
tree", Fig. 3): every worker k holds one gradient vector; the vectors are summed
element by element in reduction-tree (or parameter-server) order; the sum
drives one momentum-SGD step; the updated weights go back to every worker.
"""
import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liboracle.so")

SEG_DTYPE = np.dtype([("offset", "<u8"), ("length", "<u8"),
                      ("lr_mult", "<f4"), ("decay_mult", "<f4")])
ORDERS = {"tree": 0, "linear": 1}


class _Lib:
    """ctypes handle on one build of the oracle library."""

    def __init__(self, path):
        L = ctypes.CDLL(path)
        vp = ctypes.c_void_p
        L.orc_f16_to_f32.argtypes = [ctypes.c_uint16]
        L.orc_f16_to_f32.restype = ctypes.c_float
        L.orc_tree_reduce.argtypes = [vp, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, vp, vp]
        L.orc_sgd_step.argtypes = [vp, ctypes.c_int, vp, vp, vp, ctypes.c_float, ctypes.c_float,
                                   ctypes.c_float, ctypes.c_int]
        L.orc_broadcast.argtypes = [vp, ctypes.c_int, ctypes.c_int, vp, vp]
        L.orc_step.argtypes = [vp, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, vp, vp, vp,
                               ctypes.c_float, ctypes.c_float, ctypes.c_float, ctypes.c_int, vp, vp, vp]
        L.orc_lr_at.argtypes = [ctypes.c_int, ctypes.c_double, ctypes.c_int, ctypes.c_double, ctypes.c_int64,
                                ctypes.c_int64, ctypes.c_double, ctypes.c_int64, ctypes.c_int,
                                ctypes.POINTER(ctypes.c_float)]
        for f in ("orc_tree_reduce", "orc_sgd_step", "orc_broadcast", "orc_step", "orc_lr_at"):
            getattr(L, f).restype = ctypes.c_int
        self.L = L
        self.path = path


_default = None
_current = None


def lib():
    """The oracle library in use (liboracle.so, compiled first if missing)."""
    global _default
    if _current is not None:
        return _current.L
    if _default is None:
        if not os.path.exists(LIB_PATH):
            from . import build as _b
            _b.build()
        _default = _Lib(LIB_PATH)
    return _default.L


class use:
    """Context manager: route this module's functions through another build
    of the oracle (used by the tests that plant mistakes in a copy)."""

    def __init__(self, path):
        self.handle = _Lib(path)

    def __enter__(self):
        global _current
        self.prev, _current = _current, self.handle
        return self

    def __exit__(self, *exc):
        global _current
        _current = self.prev
        return False


def segments(segs):
    """Segment table as a C-layout structured array.  Accepts a structured
    array or a sequence of (offset, length[, lr_mult, decay_mult])."""
    if isinstance(segs, np.ndarray) and segs.dtype == SEG_DTYPE:
        return np.ascontiguousarray(segs)
    rows = []
    for s in segs:
        s = tuple(s)
        rows.append((s[0], s[1], s[2] if len(s) > 2 else 1.0, s[3] if len(s) > 3 else 1.0))
    return np.array(rows, dtype=SEG_DTYPE)


def extent(segs):
    """One past the last element any segment covers."""
    t = segments(segs)
    return int((t["offset"] + t["length"]).max()) if len(t) else 0


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def _replicas(grads):
    """List of K contiguous 1-D replicas (float32 or float16)."""
    reps = [np.ascontiguousarray(g) for g in grads]
    dt = reps[0].dtype
    if dt not in (np.float32, np.float16):
        raise TypeError("replicas must be float32 or float16")
    if any(r.dtype != dt or r.ndim != 1 for r in reps):
        raise TypeError("replicas must share one dtype and be 1-D")
    return reps, (1 if dt == np.float16 else 0)


def _ptr_table(arrays):
    return (ctypes.c_void_p * len(arrays))(*[a.ctypes.data for a in arrays])


def f16_to_f32(bits):
    """Widen binary16 bit patterns (uint16 array) to float32, one call each."""
    L = lib()
    bits = np.asarray(bits, dtype=np.uint16).ravel()
    return np.array([L.orc_f16_to_f32(int(b)) for b in bits], dtype=np.float32)


def tree_reduce(segs, grads, order="tree", out=None):
    """out[i] = sum_k grads[k][i] in the given order; untouched elements of
    `out` keep their values (zeros when `out` is not given)."""
    t = segments(segs)
    reps, dt = _replicas(grads)
    n = max(extent(t), max(len(r) for r in reps))
    if out is None:
        out = np.zeros(n, dtype=np.float32)
    tbl = _ptr_table(reps)
    rc = lib().orc_tree_reduce(_ptr(t), len(t), len(reps), dt, ORDERS[order], tbl, _ptr(out))
    if rc:
        raise ValueError(f"orc_tree_reduce failed ({rc})")
    return out


def sgd_step(segs, w, v, g, lr, mu, wd, batch):
    """Return (w', v') after one momentum-SGD step from the raw sum g."""
    t = segments(segs)
    w = np.array(w, dtype=np.float32, copy=True)
    v = np.array(v, dtype=np.float32, copy=True)
    g = np.ascontiguousarray(g, dtype=np.float32)
    rc = lib().orc_sgd_step(_ptr(t), len(t), _ptr(w), _ptr(v), _ptr(g), lr, mu, wd, int(batch))
    if rc:
        raise ValueError(f"orc_sgd_step failed ({rc})")
    return w, v


def broadcast(segs, src, dsts):
    """Copy src into every array of dsts over the segment elements, in place."""
    t = segments(segs)
    src = np.ascontiguousarray(src, dtype=np.float32)
    for d in dsts:
        assert d.dtype == np.float32 and d.flags.c_contiguous
    rc = lib().orc_broadcast(_ptr(t), len(t), len(dsts), _ptr(src), _ptr_table(dsts))
    if rc:
        raise ValueError(f"orc_broadcast failed ({rc})")
    return dsts


def step(segs, grads, w, v, lr, mu, wd, batch, order="tree", out=None, bcast=None):
    """The fused step; returns (w', v', out, bcast).  `out` and `bcast` (a list
    of K float32 arrays) are updated in place when given."""
    t = segments(segs)
    reps, dt = _replicas(grads)
    w = np.array(w, dtype=np.float32, copy=True)
    v = np.array(v, dtype=np.float32, copy=True)
    scratch = np.zeros(len(w), dtype=np.float32)
    bt = _ptr_table(bcast) if bcast is not None else None
    rc = lib().orc_step(_ptr(t), len(t), len(reps), dt, ORDERS[order], _ptr_table(reps),
                        _ptr(w), _ptr(v), lr, mu, wd, int(batch), _ptr(scratch),
                        _ptr(out) if out is not None else None, bt)
    if rc:
        raise ValueError(f"orc_step failed ({rc})")
    return w, v, out, bcast


def default_threads():
    """Host threads for step_parallel: OMP_NUM_THREADS when set (a machine
    shared between jobs sets it to each job's CPU share), else every core."""
    n = os.cpu_count() or 1
    return max(1, min(n, int(os.environ.get("OMP_NUM_THREADS", n))))


def step_parallel(segs, grads, w, v, lr, mu, wd, batch, order="tree", out=None, bcast=None, threads=None):
    """The fused step of `step`, run by `threads` host threads, each calling
    the same C function on one contiguous range of element indices.

    Every parameter's sum and update read and write only that parameter's
    element of each buffer (the workers' vectors are added element by element,
    Sec. 6.2), so cutting the index range changes no element's operations or
    their order: the result is the one `step` computes.  `grads` is a 2-D
    array (K, n) or a list of K 1-D arrays.  Returns (w', v', out, bcast) like
    `step`; `out` and the arrays of `bcast` are updated in place."""
    from concurrent.futures import ThreadPoolExecutor

    t = segments(segs)
    reps, dt = _replicas(list(grads))
    K = len(reps)
    w = np.array(w, dtype=np.float32, copy=True)
    v = np.array(v, dtype=np.float32, copy=True)
    if bcast is not None:
        for d in bcast:
            assert d.dtype == np.float32 and d.flags.c_contiguous
    n = extent(t)
    threads = threads or default_threads()
    cuts = sorted(set(n * i // threads for i in range(threads + 1)))
    L = lib()

    def addr(a, first):
        return a.ctypes.data + first * a.itemsize

    def run(a, b):
        # the segments clipped to [a, b), offsets relative to a
        rows = [(max(o, a) - a, min(o + m, b) - max(o, a), lm, dm)
                for o, m, lm, dm in zip(t["offset"].tolist(), t["length"].tolist(), t["lr_mult"].tolist(),
                                        t["decay_mult"].tolist())
                if max(o, a) < min(o + m, b)]
        if not rows:
            return 0
        sub = segments(rows)
        scratch = np.empty(b - a, dtype=np.float32)
        rt = (ctypes.c_void_p * K)(*[addr(r, a) for r in reps])
        bt = (ctypes.c_void_p * K)(*[addr(d, a) for d in bcast]) if bcast is not None else None
        return L.orc_step(_ptr(sub), len(sub), K, dt, ORDERS[order], rt, ctypes.c_void_p(addr(w, a)),
                          ctypes.c_void_p(addr(v, a)), lr, mu, wd, int(batch), _ptr(scratch),
                          ctypes.c_void_p(addr(out, a)) if out is not None else None, bt)

    with ThreadPoolExecutor(max(1, len(cuts) - 1)) as ex:
        codes = list(ex.map(lambda ab: run(*ab), zip(cuts[:-1], cuts[1:])))
    if any(codes):
        raise ValueError(f"orc_step failed ({codes})")
    return w, v, out, bcast


LR_KINDS = {"fixed": 0, "step": 1, "poly": 2}


def lr_at(kind, iter, batch, base_lr, base_batch=0, gamma=0.1, stepsize=1, max_iter=1, power=1.0):
    """Learning rate of a policy at `iter` (float32)."""
    out = ctypes.c_float()
    rc = lib().orc_lr_at(LR_KINDS[kind], base_lr, base_batch, gamma, stepsize, max_iter, power, iter, batch,
                         ctypes.byref(out))
    if rc:
        raise ValueError("invalid learning-rate policy or iteration")
    return np.float32(out.value)


def train(segs, grads, w, v, mu, wd, batch, iters, policy):
    """Steps at iterations `iters` with the policy's rate (same replicas every
    step); returns (w, v).  `policy` is a dict of lr_at keyword arguments."""
    for it in iters:
        lr = lr_at(iter=it, batch=batch, **policy)
        w, v, _, _ = step(segs, grads, w, v, float(lr), mu, wd, batch)
    return w, v

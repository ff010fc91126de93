"""ctypes binding of libfc.so (include/fc.h), argument marshalling only.

Every function here has the name of the C entry point it calls and passes
its arguments through unchanged; all computation happens in the HIP kernels
behind the C ABI.  If libfc.so is missing the import fails: there is no other
implementation to fall back to.
"""
import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("FC_LIBRARY", os.path.join(PKG, "libfc.so"))

FC_OK, FC_EINVAL, FC_EALIGN, FC_EALIAS, FC_EHIP, FC_ENOMEM, FC_ESIZE = 0, -1, -2, -3, -4, -5, -6
FC_NOALLOC_MAX_ELEMS = 16777216  # floats in the fixed raw-sum array of fc_step_noalloc
FC_F32, FC_F16 = 0, 1
FC_ORDER_TREE, FC_ORDER_LINEAR = 0, 1


class fc_segment(ctypes.Structure):
    _fields_ = [("offset", ctypes.c_uint64), ("length", ctypes.c_uint64),
                ("lr_mult", ctypes.c_float), ("decay_mult", ctypes.c_float)]


class fc_launch_opts(ctypes.Structure):
    _fields_ = [("block_threads", ctypes.c_int), ("vecs_per_thread", ctypes.c_int), ("kchunk", ctypes.c_int),
                ("max_blocks", ctypes.c_int), ("schedule", ctypes.c_int), ("k_waves", ctypes.c_int)]


class fc_plan_info(ctypes.Structure):
    _fields_ = [("K", ctypes.c_int), ("nseg", ctypes.c_int), ("dtype", ctypes.c_int), ("order", ctypes.c_int),
                ("n_elems", ctypes.c_uint64), ("extent", ctypes.c_uint64), ("ntiles", ctypes.c_int),
                ("grid", ctypes.c_int), ("block_threads", ctypes.c_int), ("vecs_per_thread", ctypes.c_int),
                ("kchunk", ctypes.c_int), ("schedule", ctypes.c_int),
                ("scratch_bytes", ctypes.c_uint64), ("k_waves", ctypes.c_int), ("lds_bytes", ctypes.c_int),
                ("rounds", ctypes.c_int)]


FC_SCHED_AUTO, FC_SCHED_FUSED, FC_SCHED_TWO_PASS, FC_SCHED_RESIDENT, FC_SCHED_RESIDENT_ONE_LAUNCH = 0, 1, 2, 3, 4
FC_KERNEL_STEP, FC_KERNEL_REDUCE, FC_KERNEL_SGD, FC_KERNEL_BCAST, FC_KERNEL_KINDS = 0, 1, 2, 3, 4
KERNEL_NAMES = ("step", "reduce", "sgd", "bcast")


class fc_timing(ctypes.Structure):
    _fields_ = [("launches", ctypes.c_int * FC_KERNEL_KINDS), ("total_us", ctypes.c_double * FC_KERNEL_KINDS)]


FC_LR_FIXED, FC_LR_STEP, FC_LR_POLY = 0, 1, 2


class fc_lr_policy(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int), ("base_batch", ctypes.c_int), ("base_lr", ctypes.c_double),
                ("gamma", ctypes.c_double), ("stepsize", ctypes.c_int64), ("max_iter", ctypes.c_int64),
                ("power", ctypes.c_double)]


if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() or "
                      "python paper_1511_00175_amd/build.py")

lib = ctypes.CDLL(LIB_PATH)

_vp = ctypes.c_void_p
_pp = ctypes.POINTER(ctypes.c_void_p)
_i, _f = ctypes.c_int, ctypes.c_float
_plan_p = ctypes.c_void_p

lib.fc_plan_create.argtypes = [ctypes.POINTER(_plan_p), ctypes.POINTER(fc_segment), _i, _i, _i, _i]
lib.fc_plan_create_ex.argtypes = [ctypes.POINTER(_plan_p), ctypes.POINTER(fc_segment), _i, _i, _i, _i,
                                  ctypes.POINTER(fc_launch_opts)]
lib.fc_plan_destroy.argtypes = [_plan_p]
lib.fc_plan_destroy.restype = None
lib.fc_tree_reduce.argtypes = [_plan_p, _pp, _vp, _vp]
lib.fc_sgd_step.argtypes = [_plan_p, _vp, _vp, _vp, _f, _f, _f, _i, _vp]
lib.fc_broadcast.argtypes = [_plan_p, _vp, _pp, _vp]
lib.fc_step.argtypes = [_plan_p, _pp, _vp, _vp, _f, _f, _f, _i, _vp, _pp, _vp]
lib.fc_step_noalloc.argtypes = [_plan_p, _pp, _vp, _vp, _f, _f, _f, _i, _vp, _pp, _vp]
lib.fc_strerror.argtypes = [_i]
lib.fc_strerror.restype = ctypes.c_char_p
lib.fc_plan_query.argtypes = [_plan_p, ctypes.POINTER(fc_plan_info)]
lib.fc_lr_at.argtypes = [ctypes.POINTER(fc_lr_policy), ctypes.c_int64, _i, ctypes.POINTER(ctypes.c_float)]
lib.fc_train.argtypes = [_plan_p, _pp, _vp, _vp, ctypes.POINTER(fc_lr_policy), ctypes.c_int64, ctypes.c_int64,
                         _f, _f, _i, _vp]
lib.fc_read_probe_blocks.argtypes = [ctypes.c_uint64]
lib.fc_read_probe_blocks.restype = ctypes.c_uint64
lib.fc_read_probe.argtypes = [_vp, ctypes.c_uint64, _vp, _vp]
lib.fc_plan_set_timing.argtypes = [_plan_p, _i]
lib.fc_plan_read_timing.argtypes = [_plan_p, ctypes.POINTER(fc_timing)]
lib.fc_plan_balance.argtypes = [_plan_p, _vp, ctypes.POINTER(ctypes.c_float), _i]
for _n in ("fc_plan_create", "fc_plan_create_ex", "fc_tree_reduce", "fc_sgd_step", "fc_broadcast", "fc_step",
           "fc_step_noalloc",
           "fc_plan_query", "fc_plan_set_timing", "fc_plan_read_timing", "fc_lr_at", "fc_train",
           "fc_read_probe", "fc_plan_balance"):
    getattr(lib, _n).restype = ctypes.c_int


class FcError(RuntimeError):
    def __init__(self, fn, code):
        self.code = code
        super().__init__(f"{fn}: {fc_strerror(code)} ({code})")


def _check(fn, rc):
    if rc != FC_OK:
        raise FcError(fn, rc)
    return rc


def _ptr_array(ptrs):
    """A C array of device pointers from a sequence of ints (a ctypes array
    passes through unchanged)."""
    if ptrs is None or isinstance(ptrs, ctypes.Array):
        return ptrs
    return (ctypes.c_void_p * len(ptrs))(*[int(p) for p in ptrs])


def segment_array(rows):
    """fc_segment[] from (offset, length[, lr_mult, decay_mult]) rows."""
    rows = list(rows)
    arr = (fc_segment * max(len(rows), 1))()
    for i, r in enumerate(rows):
        r = tuple(r)
        arr[i] = fc_segment(int(r[0]), int(r[1]), float(r[2]) if len(r) > 2 else 1.0,
                            float(r[3]) if len(r) > 3 else 1.0)
    return arr, len(rows)


def fc_strerror(code):
    return lib.fc_strerror(int(code)).decode()


def fc_plan_create(segs, K, gdt=FC_F32, order=FC_ORDER_TREE, opts=None):
    """Returns (rc, plan handle).  `opts` is a dict of fc_launch_opts fields."""
    arr, n = segment_array(segs)
    h = _plan_p()
    if opts is None:
        rc = lib.fc_plan_create(ctypes.byref(h), arr, n, int(K), int(gdt), int(order))
    else:
        o = fc_launch_opts(0, 0, 0, 0, 0, 0)
        fields = [f[0] for f in fc_launch_opts._fields_]
        for k, v in opts.items():
            if k not in fields:  # a ctypes structure would keep it as a plain attribute
                raise ValueError(f"unknown launch option {k!r} (fields: {', '.join(fields)})")
            setattr(o, k, int(v))
        rc = lib.fc_plan_create_ex(ctypes.byref(h), arr, n, int(K), int(gdt), int(order), ctypes.byref(o))
    return rc, h


def fc_plan_destroy(plan):
    lib.fc_plan_destroy(plan)


def fc_plan_query(plan):
    info = fc_plan_info()
    _check("fc_plan_query", lib.fc_plan_query(plan, ctypes.byref(info)))
    return info


def fc_plan_set_timing(plan, enable):
    return lib.fc_plan_set_timing(plan, 1 if enable else 0)


def fc_plan_read_timing(plan):
    """{kernel name: (launches, total us)} since the previous read."""
    t = fc_timing()
    _check("fc_plan_read_timing", lib.fc_plan_read_timing(plan, ctypes.byref(t)))
    return {KERNEL_NAMES[i]: (t.launches[i], t.total_us[i]) for i in range(FC_KERNEL_KINDS)}


N_XCD_RATES = 16


def fc_plan_balance(plan, stream=0):
    """Returns (rc, [relative rate of XCD x for x < 16], 0 where no block ran)."""
    rates = (ctypes.c_float * N_XCD_RATES)()
    rc = lib.fc_plan_balance(plan, stream, rates, N_XCD_RATES)
    return rc, list(rates)


def fc_tree_reduce(plan, grads, out, stream=0):
    return lib.fc_tree_reduce(plan, _ptr_array(grads), out, stream)


def fc_sgd_step(plan, w, v, g, lr, mu, wd, batch, stream=0):
    return lib.fc_sgd_step(plan, w, v, g, lr, mu, wd, int(batch), stream)


def fc_broadcast(plan, src, dst, stream=0):
    return lib.fc_broadcast(plan, src, _ptr_array(dst), stream)


def fc_step(plan, grads, w, v, lr, mu, wd, batch, out=None, bcast_dst=None, stream=0):
    return lib.fc_step(plan, _ptr_array(grads), w, v, lr, mu, wd, int(batch), out, _ptr_array(bcast_dst), stream)


def fc_step_noalloc(plan, grads, w, v, lr, mu, wd, batch, out=None, bcast_dst=None, stream=0):
    return lib.fc_step_noalloc(plan, _ptr_array(grads), w, v, lr, mu, wd, int(batch), out, _ptr_array(bcast_dst),
                               stream)


_LR_KINDS = {"fixed": FC_LR_FIXED, "step": FC_LR_STEP, "poly": FC_LR_POLY}


def lr_policy(kind, base_lr, base_batch=0, gamma=0.1, stepsize=1, max_iter=1, power=1.0):
    """fc_lr_policy from keyword arguments (kind: "fixed", "step" or "poly")."""
    return fc_lr_policy(_LR_KINDS[kind], int(base_batch), float(base_lr), float(gamma), int(stepsize),
                        int(max_iter), float(power))


def fc_lr_at(policy, iter, batch):
    """Returns (rc, lr)."""
    out = ctypes.c_float()
    rc = lib.fc_lr_at(ctypes.byref(policy) if policy is not None else None, int(iter), int(batch),
                      ctypes.byref(out))
    return rc, out.value


def fc_train(plan, grads, w, v, policy, first_iter, n_iters, mu, wd, batch, stream=0):
    return lib.fc_train(plan, _ptr_array(grads), w, v, ctypes.byref(policy), int(first_iter), int(n_iters),
                        mu, wd, int(batch), stream)


def fc_read_probe_blocks(nbytes):
    return lib.fc_read_probe_blocks(int(nbytes))


def fc_read_probe(src, nbytes, out, stream=0):
    return lib.fc_read_probe(src, int(nbytes), out, stream)

"""MI355X (gfx950) gradient aggregation + momentum SGD, after FireCaffe
(Iandola et al., arXiv 1511.00175): K workers' gradient replicas resident in
device memory are summed in binary reduction-tree order (Sec. 6.2, Fig. 3b) or
parameter-server order (Sec. 6.1, Fig. 3a), averaged over the batch, applied as
momentum SGD with weight decay, and the updated weights are optionally sent
back to every worker (Fig. 3 caption).

The work is done by HIP kernels behind the C ABI of include/fc.h; this package
only marshals torch tensors (device memory and the current stream) into it.
"""
import weakref

from . import _fc
from ._fc import (FC_F16, FC_F32, FC_NOALLOC_MAX_ELEMS, FC_ORDER_LINEAR, FC_ORDER_TREE, FC_SCHED_AUTO,  # noqa: F401
                  FC_SCHED_FUSED, FC_SCHED_RESIDENT, FC_SCHED_RESIDENT_ONE_LAUNCH, FC_SCHED_TWO_PASS, FcError,
                  fc_broadcast, fc_plan_create, fc_plan_destroy, fc_plan_query, fc_lr_at, fc_plan_balance,
                  fc_plan_read_timing, fc_plan_set_timing, fc_read_probe, fc_read_probe_blocks, fc_sgd_step, fc_step,
                  fc_step_noalloc, fc_strerror, fc_train, fc_tree_reduce, lr_policy)

__all__ = ["Plan", "FcError", "fc_plan_create", "fc_plan_destroy", "fc_plan_query", "fc_plan_set_timing",
           "fc_plan_read_timing", "fc_plan_balance", "fc_tree_reduce", "fc_sgd_step", "fc_broadcast", "fc_step",
           "fc_step_noalloc", "fc_strerror",
           "fc_lr_at", "fc_train", "lr_policy", "lr_at", "fc_read_probe", "fc_read_probe_blocks", "read_probe"]


def lr_at(iter, batch, **policy):
    """Learning rate of a policy (lr_policy keyword arguments) at `iter`."""
    rc, lr = fc_lr_at(lr_policy(**policy), iter, batch)
    if rc:
        raise FcError("fc_lr_at", rc)
    return lr

def read_probe(src, out, stream=None):
    """Streaming read of the whole tensor `src` (fc_read_probe); `out` is an
    fp32 tensor of at least fc_read_probe_blocks(src bytes) elements on the
    same device."""
    import torch
    if not isinstance(src, torch.Tensor) or src.device.type != "cuda" or not src.is_contiguous():
        raise ValueError("src must be a contiguous device tensor")
    nbytes = src.numel() * src.element_size()
    _check_vector(out, "out", "float32", src.device, fc_read_probe_blocks(nbytes))
    rc = fc_read_probe(src.data_ptr(), nbytes, out.data_ptr(), _stream(stream))
    if rc:
        raise FcError("fc_read_probe", rc)


_DTYPES = {"f32": FC_F32, "f16": FC_F16}
_ORDERS = {"tree": FC_ORDER_TREE, "linear": FC_ORDER_LINEAR}


_CURRENT_STREAM = None  # torch's current-stream handle of the current device, looked up once


def _stream(stream):
    """The HIP stream handle of a call: the given stream (a torch stream or a
    handle), else torch's current stream on the current device.  The latter
    is read through torch's raw accessors: building a torch Stream object per
    call costs more host time (about 2.7 us on MI355X's host) than a small
    step's kernel takes on the GPU."""
    global _CURRENT_STREAM
    if stream is not None:
        return int(stream) if not hasattr(stream, "cuda_stream") else stream.cuda_stream
    if _CURRENT_STREAM is None:
        import torch
        raw = getattr(torch._C, "_cuda_getCurrentRawStream", None)
        dev = getattr(torch._C, "_cuda_getDevice", None)
        if raw is not None and dev is not None:
            _CURRENT_STREAM = lambda: raw(dev())  # noqa: E731
        else:  # a torch without the raw accessors: the public, slower call
            _CURRENT_STREAM = lambda: torch.cuda.current_stream().cuda_stream  # noqa: E731
    return _CURRENT_STREAM()


def _ptr(t):
    return None if t is None else t.data_ptr()


def _rows(x):
    """Device pointers of the K replicas: a list of tensors or the rows of a
    2-D tensor (K, stride)."""
    if isinstance(x, (list, tuple)):
        return [t.data_ptr() for t in x]
    if x.dim() != 2 or x.stride(1) != 1:
        raise ValueError("replicas must be a list of tensors or a row-major 2-D tensor")
    base, step = x.data_ptr(), x.stride(0) * x.element_size()
    return [base + k * step for k in range(x.shape[0])]


_TORCH_DTYPES = {"f32": "float32", "f16": "float16"}


_STEP_CACHE = 64  # sets of step buffers whose checks are kept per plan


def _sig(x):
    """What a tensor's checks depend on and `.data` assignment or set_() can
    change in place: address, shape, strides, dtype, device."""
    return (x.data_ptr(), x.shape, x.stride(), x.dtype, x.get_device())


def _check_vector(t, name, dtype, device, n):
    """`t` must be a contiguous torch tensor of `dtype` on `device` holding at
    least n elements (the C ABI sees only the pointer, so a short or
    mistyped buffer would be read or written out of bounds on the GPU)."""
    import torch
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name} must be a torch tensor")
    if t.dtype != getattr(torch, dtype):
        raise ValueError(f"{name} must be {dtype}, not {t.dtype}")
    if t.device != device:
        raise ValueError(f"{name} is on {t.device}, the plan on {device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.numel() < n:
        raise ValueError(f"{name} holds {t.numel()} elements, the plan covers {n}")


class Plan:
    """One segment table and worker count (fc_plan).

    segments: rows (offset, length[, lr_mult, decay_mult]) in elements.
    dtype   : replica storage, "f32" or "f16".
    order   : "tree" (reduction tree) or "linear" (parameter server).
    opts    : launch shape (block_threads, vecs_per_thread, kchunk,
              max_blocks, k_waves) and fc_step schedule (0 auto, 1 fused,
              2 two-pass, 3 resident, 4 resident with every round in one
              launch); results do not depend on them.
    """

    _step_cache = None  # {buffer ids: (weak references, signatures, checked pointers)}

    def __init__(self, segments, K, dtype="f32", order="tree", **opts):
        import torch
        rc, h = fc_plan_create(segments, K, _DTYPES[dtype], _ORDERS[order], opts or None)
        if rc:
            raise FcError("fc_plan_create", rc)
        self.handle = h
        self.K = K
        self.dtype = dtype
        self.order = order
        # what every buffer passed to the plan must cover, and where
        self.extent = fc_plan_query(h).extent
        self.device = torch.device("cuda", torch.cuda.current_device())

    def _cached(self, role, x, check, *args):
        """check(x, *args) -- the checked pointer(s) of buffer x in `role` --
        done once per tensor: while a call passes the tensor object the
        previous call passed in this role (held by weak reference), with the
        same address, shape, strides, dtype and device (all of which `.data`
        assignment or set_() can change in place), the previous result is
        reused."""
        if type(x).__name__ not in ("Tensor", "Parameter"):
            return check(x, *args)
        cache = self.__dict__.setdefault("_checked", {})
        sig = _sig(x)
        hit = cache.get(role)
        if hit is not None and hit[0]() is x and hit[1] == sig:
            return hit[2]
        got = check(x, *args)
        cache[role] = (weakref.ref(x), sig, got)
        return got

    def _vec_checked(self, t, name):
        _check_vector(t, name, "float32", self.device, self.extent)
        return t.data_ptr()

    def _vec(self, t, name, optional=False):
        """Pointer of an fp32 buffer (w, v, out, g, src) after checking it."""
        if t is None and optional:
            return None
        return self._cached(name, t, self._vec_checked, name)

    def _reps(self, x, name, dtype):
        """Pointers of K buffers (replicas of the plan's type, or fp32
        broadcast destinations), as a C array: a list of K tensors or a 2-D
        tensor of K rows, each checked like _vec."""
        if isinstance(x, (list, tuple)):
            if len(x) != self.K:
                raise ValueError(f"{name}: {len(x)} buffers for a plan of K={self.K}")
            for k, t in enumerate(x):
                _check_vector(t, f"{name}[{k}]", dtype, self.device, self.extent)
            return _fc._ptr_array([t.data_ptr() for t in x])
        return self._cached(name, x, self._rows_checked, name, dtype)

    def _rows_checked(self, x, name, dtype):
        import torch
        if not isinstance(x, torch.Tensor) or x.dim() != 2:
            raise ValueError(f"{name} must be a list of K tensors or a 2-D tensor of K rows")
        if x.shape[0] != self.K:
            raise ValueError(f"{name} has {x.shape[0]} rows for a plan of K={self.K}")
        if x.stride(1) != 1 or (self.K > 1 and x.stride(0) < x.shape[1]):
            raise ValueError(f"{name} must be row-major with rows that do not overlap")
        if x.shape[1] < self.extent:
            raise ValueError(f"{name} rows hold {x.shape[1]} elements, the plan covers {self.extent}")
        if x.dtype != getattr(torch, dtype):
            raise ValueError(f"{name} must be {dtype}, not {x.dtype}")
        if x.device != self.device:
            raise ValueError(f"{name} is on {x.device}, the plan on {self.device}")
        return _fc._ptr_array(_rows(x))

    def _grads(self, x):
        return self._reps(x, "grads", _TORCH_DTYPES[self.dtype])

    def close(self):
        """Free the plan (fc_plan_destroy).  Kernels queued by earlier calls
        may still read its device tables, so the plan's device is
        synchronized first; garbage collection of a Plan calls this too."""
        if self.handle:
            try:
                import torch
                torch.cuda.synchronize(self.device)
            except Exception:
                pass
            fc_plan_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def info(self):
        return fc_plan_query(self.handle)

    def set_timing(self, enable=True):
        rc = fc_plan_set_timing(self.handle, enable)
        if rc:
            raise FcError("fc_plan_set_timing", rc)

    def read_timing(self):
        """{kernel: (launches, total us)} since the previous read."""
        return fc_plan_read_timing(self.handle)

    def balance(self, stream=None):
        """Re-divide the resident schedule's tiles by the per-XCD rates of the
        last launch (fc_plan_balance); returns the rates (relative to the
        mean, 0 for XCDs that ran no block)."""
        rc, rates = fc_plan_balance(self.handle, _stream(stream))
        if rc:
            raise FcError("fc_plan_balance", rc)
        return rates

    def tree_reduce(self, grads, out, stream=None):
        rc = fc_tree_reduce(self.handle, self._grads(grads), self._vec(out, "out"), _stream(stream))
        if rc:
            raise FcError("fc_tree_reduce", rc)

    def sgd_step(self, w, v, g, lr, mu, wd, batch, stream=None):
        rc = fc_sgd_step(self.handle, self._vec(w, "w"), self._vec(v, "v"), self._vec(g, "g"), lr, mu, wd, batch,
                         _stream(stream))
        if rc:
            raise FcError("fc_sgd_step", rc)

    def broadcast(self, src, dst, stream=None):
        rc = fc_broadcast(self.handle, self._vec(src, "src"), self._reps(dst, "dst", "float32"), _stream(stream))
        if rc:
            raise FcError("fc_broadcast", rc)

    def train(self, grads, w, v, policy, first_iter, n_iters, mu, wd, batch, stream=None):
        """n_iters fused steps with the policy's rate (policy: lr_policy
        keyword arguments); the same replicas feed every step."""
        rc = fc_train(self.handle, self._grads(grads), self._vec(w, "w"), self._vec(v, "v"), lr_policy(**policy),
                      first_iter, n_iters, mu, wd, batch, _stream(stream))
        if rc:
            raise FcError("fc_train", rc)

    def _step_args(self, grads, w, v, out, bcast):
        """Checked pointers of a step's buffers.  The results of the last
        _STEP_CACHE distinct sets of tensors are kept (by weak reference, with
        each tensor's address, shape, strides, dtype and device), so that
        steps that cycle through a few sets of buffers -- double-buffered
        gradients, rotating weights -- are checked once per set; any other
        call checks every buffer (_vec, _reps)."""
        key = (id(grads), id(w), id(v), id(out), id(bcast))
        cache = self._step_cache
        hit = cache.get(key) if cache is not None else None
        if hit is not None:
            refs, sigs, got = hit
            if (refs[0]() is grads and refs[1]() is w and refs[2]() is v
                    and (out is None if refs[3] is None else refs[3]() is out)
                    and (bcast is None if refs[4] is None else refs[4]() is bcast)
                    and sigs == (_sig(grads), _sig(w), _sig(v), out is not None and _sig(out),
                                 bcast is not None and _sig(bcast))):
                return got
        got = (self._grads(grads), self._vec(w, "w"), self._vec(v, "v"), self._vec(out, "out", optional=True),
               None if bcast is None else self._reps(bcast, "bcast", "float32"))
        bufs = (grads, w, v, out, bcast)
        if all(b is None or type(b).__name__ in ("Tensor", "Parameter") for b in bufs) and grads is not None:
            if cache is None or len(cache) >= _STEP_CACHE:
                cache = self._step_cache = {}
            cache[key] = (tuple(None if b is None else weakref.ref(b) for b in bufs),
                          (_sig(grads), _sig(w), _sig(v), out is not None and _sig(out),
                           bcast is not None and _sig(bcast)), got)
        return got

    def step(self, grads, w, v, lr, mu, wd, batch, out=None, bcast=None, stream=None):
        g, wp, vp, op, bp = self._step_args(grads, w, v, out, bcast)
        rc = fc_step(self.handle, g, wp, vp, lr, mu, wd, batch, op, bp, _stream(stream))
        if rc:
            raise FcError("fc_step", rc)

    def step_noalloc(self, grads, w, v, lr, mu, wd, batch, out=None, bcast=None, stream=None):
        """fc_step_noalloc: the step in two passes with the raw sum in the
        library's fixed device array (no allocation)."""
        g, wp, vp, op, bp = self._step_args(grads, w, v, out, bcast)
        rc = fc_step_noalloc(self.handle, g, wp, vp, lr, mu, wd, batch, op, bp, _stream(stream))
        if rc:
            raise FcError("fc_step_noalloc", rc)

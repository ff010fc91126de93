"""The torch binding checks every buffer against the plan before it calls the
C ABI, which sees only pointers: K replicas (or K rows) of the plan's type,
fp32 w, v, out, g, src and destinations, each contiguous, on the plan's
device and covering the plan's extent.  A wrong buffer raises ValueError
before anything reaches the library; a right one reaches it (here a plan
without a device handle, which the library refuses with FC_EINVAL)."""
import pytest

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def fc():
    import paper_1511_00175_amd as m
    return m


def fake_plan(fc, K=4, dtype="f32", extent=1000, device="cpu"):
    """A Plan object with the facts the checks read and no library plan."""
    p = object.__new__(fc.Plan)
    p.handle, p.K, p.dtype, p.order, p.extent, p.device = None, K, dtype, "tree", extent, torch.device(device)
    return p


def bufs(K=4, n=1000, gdt=torch.float32):
    return (torch.zeros((K, n + 64), dtype=gdt), torch.zeros(n), torch.zeros(n), torch.zeros(n),
            torch.zeros((K, n)))


def reaches_library(fc, call):
    with pytest.raises(fc.FcError) as e:
        call()
    assert e.value.code == fc._fc.FC_EINVAL


def test_valid_buffers_reach_the_library(fc):
    p = fake_plan(fc)
    r, w, v, out, dst = bufs()
    reaches_library(fc, lambda: p.step(r, w, v, 0.1, 0.9, 0.0, 1, stream=0))
    reaches_library(fc, lambda: p.step(list(r), w, v, 0.1, 0.9, 0.0, 1, out=out, bcast=dst, stream=0))
    reaches_library(fc, lambda: p.step_noalloc(r, w, v, 0.1, 0.9, 0.0, 1, bcast=list(dst), stream=0))
    reaches_library(fc, lambda: p.tree_reduce(r[:, :1000], out, stream=0))
    reaches_library(fc, lambda: p.sgd_step(w, v, out, 0.1, 0.9, 0.0, 1, stream=0))
    reaches_library(fc, lambda: p.broadcast(out, dst, stream=0))
    h = fake_plan(fc, dtype="f16")
    reaches_library(fc, lambda: h.step(bufs(gdt=torch.float16)[0], w, v, 0.1, 0.9, 0.0, 1, stream=0))


@pytest.mark.parametrize("case", [
    "few_replicas", "many_rows", "replica_dtype", "short_rows", "short_replica", "overlapping_rows",
    "short_w", "w_dtype", "strided_v", "short_out", "bcast_dtype", "few_dsts", "wrong_device", "not_tensor",
])
def test_wrong_buffers_raise_before_the_library(fc, case):
    p = fake_plan(fc)
    r, w, v, out, dst = bufs()
    kw = {}
    if case == "few_replicas":
        r = list(r)[:3]
    elif case == "many_rows":
        r = torch.zeros((5, 1064))
    elif case == "replica_dtype":
        r = r.half()
    elif case == "short_rows":
        r = r[:, :999]
    elif case == "short_replica":
        r = [t for t in r[:3]] + [torch.zeros(999)]
    elif case == "overlapping_rows":
        r = torch.zeros(2000).as_strided((4, 1000), (10, 1))
    elif case == "short_w":
        w = w[:999]
    elif case == "w_dtype":
        w = w.double()
    elif case == "strided_v":
        v = torch.zeros(2000)[::2]
    elif case == "short_out":
        kw["out"] = out[:10]
    elif case == "bcast_dtype":
        kw["bcast"] = dst.half()
    elif case == "few_dsts":
        kw["bcast"] = list(dst)[:2]
    elif case == "wrong_device":
        p = fake_plan(fc, device="cuda:0")
    elif case == "not_tensor":
        w = w.data_ptr()
    with pytest.raises(ValueError):
        p.step(r, w, v, 0.1, 0.9, 0.0, 1, stream=0, **kw)


def test_other_calls_check_their_buffers(fc):
    p = fake_plan(fc)
    r, w, v, out, dst = bufs()
    with pytest.raises(ValueError):
        p.tree_reduce(r, out[:5])
    with pytest.raises(ValueError):
        p.sgd_step(w, v, out.half(), 0.1, 0.9, 0.0, 1)
    with pytest.raises(ValueError):
        p.broadcast(out, dst[:, :10])
    with pytest.raises(ValueError):
        p.train(r.half(), w, v, dict(kind="fixed", base_lr=0.1), 0, 1, 0.9, 0.0, 1)
    with pytest.raises(ValueError):
        p.step_noalloc(r, w, v[:3], 0.1, 0.9, 0.0, 1)


def test_a_tensor_changed_in_place_is_checked_again(fc):
    """The per-role check cache keys on the tensor's address, shape, strides,
    dtype and device: a tensor whose storage is swapped in place (.data
    assignment, set_) is checked again, even when its address is reused."""
    p = fake_plan(fc)
    r, w, v, out, dst = bufs()
    reaches_library(fc, lambda: p.step(r, w, v, 0.1, 0.9, 0.0, 1, stream=0))
    reaches_library(fc, lambda: p.step(r, w, v, 0.1, 0.9, 0.0, 1, stream=0))  # cached
    w.data = torch.zeros(1000, dtype=torch.float64)
    with pytest.raises(ValueError):
        p.step(r, w, v, 0.1, 0.9, 0.0, 1, stream=0)
    w.data = torch.zeros(1000)
    reaches_library(fc, lambda: p.step(r, w, v, 0.1, 0.9, 0.0, 1, stream=0))
    w.set_(torch.zeros(10))
    with pytest.raises(ValueError):
        p.step(r, w, v, 0.1, 0.9, 0.0, 1, stream=0)
    # a row tensor reshaped in place
    w.set_(torch.zeros(1000))
    r.set_(torch.zeros((4, 500)))
    with pytest.raises(ValueError):
        p.step(r, w, v, 0.1, 0.9, 0.0, 1, stream=0)


def test_read_probe_checks_its_buffers(fc):
    with pytest.raises(ValueError):
        fc.read_probe(torch.zeros(4096), torch.zeros(16), stream=0)  # host tensor
    with pytest.raises(ValueError):
        fc.read_probe(torch.zeros(8192)[::2], torch.zeros(16), stream=0)


def test_unknown_launch_option_is_refused(fc):
    with pytest.raises(ValueError):
        fc._fc.fc_plan_create([(0, 1000)], 4, opts=dict(block=64))


def test_rotating_buffers_are_each_checked(fc):
    """Steps that cycle through several sets of buffers reuse each set's
    checks; a tensor created after another was freed (and that may take its
    id) is checked on its own."""
    import gc
    p = fake_plan(fc)
    sets = [bufs()[:3] for _ in range(3)]
    for _ in range(2):
        for r, w, v in sets:
            reaches_library(fc, lambda: p.step(r, w, v, 0.1, 0.9, 0.0, 1, stream=0))
    r, w, v = sets[1]
    del sets, w
    gc.collect()
    for _ in range(50):  # new tensors, some of which reuse freed ids
        short = torch.zeros(999)
        with pytest.raises(ValueError):
            p.step(r, short, v, 0.1, 0.9, 0.0, 1, stream=0)

"""Learning-rate policies: the library's host function against the oracle's,
bit for bit, and argument errors (no GPU needed)."""
import numpy as np
import pytest

import oracle


@pytest.fixture(scope="module")
def fc():
    import paper_1511_00175_amd as m
    return m


def policies(rng):
    yield dict(kind="fixed", base_lr=0.01)
    yield dict(kind="fixed", base_lr=0.01, base_batch=256)
    yield dict(kind="step", base_lr=0.01, gamma=0.1, stepsize=10)
    yield dict(kind="step", base_lr=0.04, gamma=0.1, stepsize=7, base_batch=256)
    yield dict(kind="poly", base_lr=0.08, max_iter=97, power=0.5)
    yield dict(kind="poly", base_lr=0.01, max_iter=50, power=0.5, base_batch=32)
    for _ in range(20):
        yield dict(kind="poly", base_lr=float(rng.uniform(0, 1)), max_iter=int(rng.integers(1, 1000)),
                   power=float(rng.uniform(0, 3)), base_batch=int(rng.integers(0, 2048)))
        yield dict(kind="step", base_lr=float(rng.uniform(0, 1)), gamma=float(rng.uniform(0.01, 2)),
                   stepsize=int(rng.integers(1, 100)), base_batch=int(rng.integers(0, 2048)))


def test_library_matches_oracle(fc):
    rng = np.random.default_rng(11)
    for pol in policies(rng):
        top = pol.get("max_iter", 500)
        for it in sorted(set([0, 1, top // 2, top] + list(rng.integers(0, top + 1, 20)))):
            for batch in (1, 32, 256, 1024):
                want = oracle.lr_at(iter=int(it), batch=batch, **pol)
                got = np.float32(fc.lr_at(int(it), batch, **pol))
                assert got.view(np.uint32) == want.view(np.uint32), (pol, it, batch)


def test_invalid_policies(fc):
    f = fc._fc
    bad = [(f.lr_policy("poly", 0.1, max_iter=10), 11, 32), (f.lr_policy("poly", 0.1, max_iter=0), 0, 32),
           (f.lr_policy("step", 0.1, stepsize=0), 1, 32), (f.lr_policy("step", 0.1, gamma=0.0), 1, 32),
           (f.lr_policy("fixed", -0.1), 0, 32), (f.lr_policy("fixed", 0.1), -1, 32),
           (f.lr_policy("fixed", 0.1), 0, 0), (f.lr_policy("fixed", 0.1, base_batch=-1), 0, 32)]
    for pol, it, batch in bad:
        assert f.fc_lr_at(pol, it, batch)[0] == f.FC_EINVAL
    assert f.fc_lr_at(None, 0, 32)[0] == f.FC_EINVAL
    assert f.lib.fc_train(None, None, None, None, None, 0, 1, 0.9, 0.0, 32, None) == f.FC_EINVAL

"""Multi-step driver: fc_train over many iterations with the learning-rate
policies of Sec. 7.2 (step, batch scaling) and Sec. 7.3 (poly 0.5) against
the oracle running the same steps, bit for bit."""
import numpy as np
import pytest

import oracle
from gpu_cases import host_replicas, same_bits, to_dev
from workloads import gen

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def fc(device):
    import paper_1511_00175_amd as m
    return m


POLICIES = [dict(kind="step", base_lr=0.01, gamma=0.1, stepsize=10, base_batch=256),
            dict(kind="poly", base_lr=0.08, max_iter=40, power=0.5),
            dict(kind="fixed", base_lr=0.04)]


# K, replica type, fc_step schedule (fused, two passes, resident)
@pytest.mark.parametrize("K,dtype,schedule", [(5, "f32", 1), (70, "f32", 2), (9, "f16", 3), (33, "f32", 3)])
@pytest.mark.parametrize("pi", range(len(POLICIES)))
def test_train_matches_oracle(fc, K, dtype, schedule, pi):
    import torch
    pol = POLICIES[pi]
    rng = np.random.default_rng(K * 10 + pi)
    rows, ext = gen.random_table(rng, 4, 1500, 4)
    n = (ext + 7) // 8 * 8 + 64  # 16-byte aligned fp16 and fp32 rows
    reps = host_replicas(rng, K, n, np.float16 if dtype == "f16" else np.float32, scale=0.01)
    w = (rng.standard_normal(n) * 0.05).astype(np.float32)
    v = np.zeros(n, np.float32)
    batch = 1024
    ew, ev = oracle.train(rows, list(reps), w, v, 0.9, 5e-4, batch, range(40), pol)
    plan = fc.Plan(rows, K, dtype, "tree", schedule=schedule)
    w_d, v_d = to_dev(w), to_dev(v)
    r_d = to_dev(reps)
    plan.train(r_d, w_d, v_d, pol, 0, 25, 0.9, 5e-4, batch)   # iterations 0..24
    plan.train(r_d, w_d, v_d, pol, 25, 15, 0.9, 5e-4, batch)  # then 25..39
    torch.cuda.synchronize()
    assert same_bits(w_d.cpu().numpy(), ew) == 0 and same_bits(v_d.cpu().numpy(), ev) == 0
    plan.close()


def test_train_rejects_a_schedule_past_its_end(fc):
    import torch
    plan = fc.Plan([(0, 100, 1, 1)], 2, "f32", "tree")
    x = torch.zeros((2, 128), device="cuda")
    w, v = torch.ones(128, device="cuda"), torch.zeros(128, device="cuda")
    with pytest.raises(fc.FcError):
        plan.train(x, w, v, dict(kind="poly", base_lr=0.1, max_iter=10), 5, 10, 0.9, 0.0, 32)
    torch.cuda.synchronize()
    assert float(w.sum()) == 128.0  # nothing was enqueued


@pytest.mark.parametrize("schedule", [1, 3])
def test_checkpoint_resume_is_bit_exact(fc, tmp_path, schedule):
    """Training state is (w, v, iteration): a run stopped after iteration 17,
    its w and v written to disk (torch.save) and loaded back into new device
    tensors with a new plan (weights_only load), continues to the same bits as
    an uninterrupted run, and both equal the oracle's 30 steps (the step is
    deterministic, so resuming needs nothing else)."""
    import torch
    pol = POLICIES[0]
    rng = np.random.default_rng(17 + schedule)
    rows, ext = gen.random_table(rng, 5, 3000, 4)
    n = (ext + 7) // 8 * 8 + 64
    K = 12
    reps = host_replicas(rng, K, n, np.float32, scale=0.01)
    w = (rng.standard_normal(n) * 0.05).astype(np.float32)
    v = np.zeros(n, np.float32)
    ew, ev = oracle.train(rows, list(reps), w, v, 0.9, 5e-4, 256, range(30), pol)
    r_d = to_dev(reps)
    # uninterrupted
    plan = fc.Plan(rows, K, "f32", "tree", schedule=schedule)
    wa, va = to_dev(w), to_dev(v)
    plan.train(r_d, wa, va, pol, 0, 30, 0.9, 5e-4, 256)
    torch.cuda.synchronize()
    plan.close()
    # interrupted after iteration 17, state through a file
    plan = fc.Plan(rows, K, "f32", "tree", schedule=schedule)
    wb, vb = to_dev(w), to_dev(v)
    plan.train(r_d, wb, vb, pol, 0, 18, 0.9, 5e-4, 256)
    torch.cuda.synchronize()
    plan.close()
    path = tmp_path / "state.pt"
    torch.save({"w": wb.cpu(), "v": vb.cpu(), "iter": 18}, path)
    del wb, vb
    state = torch.load(path, weights_only=True)
    wc, vc = state["w"].cuda(), state["v"].cuda()
    plan = fc.Plan(rows, K, "f32", "tree", schedule=schedule)
    plan.train(r_d, wc, vc, pol, state["iter"], 30 - state["iter"], 0.9, 5e-4, 256)
    torch.cuda.synchronize()
    plan.close()
    assert torch.equal(wa.view(torch.int32), wc.view(torch.int32))
    assert torch.equal(va.view(torch.int32), vc.view(torch.int32))
    assert same_bits(wc.cpu().numpy(), ew) == 0 and same_bits(vc.cpu().numpy(), ev) == 0

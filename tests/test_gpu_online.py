"""The online step (m = 1, squared error, Algorithm 2) as one launch with a bounded grid
barrier, against the fp64 dense oracle, and against the general step path
(LST_OPT_ONLINE_KERNEL = 0) on the same inputs.

Tolerances as for every step: relative 1e-4 on the loss and grad_h of the first step, 1e-3
after; bit-exact untouched rows of V; state bit-identical after a rejected step.
"""
import numpy as np
import pytest
import torch

import paper_1606_08061_amd as lst
from gpu_common import DEV, make_factored, oracle_step, rel, to_dev
from workloads import LOSS_SQUARED, Stream, Workload

pytestmark = pytest.mark.gpu

TOL1 = 1e-4
TOL100 = 1e-3


def _run(w, steps, general=False, batches=None):
    s = Stream(w)
    f = make_factored(w, s.V0)
    if general:
        f.set_option(lst.LST_OPT_ONLINE_KERNEL, 0)
    W = s.V0.astype(np.float64)
    f.profile(True)
    for t in range(steps):
        H, idx, val = batches[t] if batches else s.batch()
        ref = oracle_step(W, H, idx, val, w)
        loss, g = f.step(*to_dev(H, idx, val), w.lr)
        assert f.sync_status() == 0
        tol = TOL1 if t == 0 else TOL100
        assert abs(loss.item() - ref.loss) <= tol * abs(ref.loss) + 1e-12, t
        assert rel(g.cpu().numpy(), ref.grad_H) <= tol, t
        W = ref.W_new
    prof = f.profile_read()
    Wg = f.materialize_W().cpu().numpy()
    f.close()
    return Wg, W, prof


@pytest.mark.parametrize("D,d,K", [(3000, 64, 5), (20000, 500, 5), (5000, 33, 1), (800, 1, 2),
                                   (4000, 1030, 3), (2000, 96, 0)])
def test_online_kernel_matches_oracle(D, d, K):
    w = Workload("t", LOSS_SQUARED, D, d, 1, K, index_dist="zipf", lr=0.01)
    Wg, W, prof = _run(w, 40)
    assert rel(Wg, W) <= TOL100
    assert prof["online"][0] == 40 and prof["contract"][0] == 0  # the fused launch ran


def test_online_kernel_and_general_path_agree():
    w = Workload("t", LOSS_SQUARED, 6000, 128, 1, 4, index_dist="zipf")
    s = Stream(w)
    batches = [s.batch() for _ in range(30)]
    Wa, W, pa = _run(w, 30, batches=batches)
    Wb, _, pb = _run(w, 30, general=True, batches=batches)
    assert pa["online"][0] == 30 and pb["online"][0] == 0 and pb["contract"][0] == 30
    assert rel(Wa, W) <= TOL100 and rel(Wb, W) <= TOL100 and rel(Wa, Wb) <= TOL100


def test_online_mixed_with_minibatches():
    # m = 1 steps between m = 16 steps: the two-stream counters and the online barrier
    # counter stay consistent
    w = Workload("t", LOSS_SQUARED, 4000, 48, 16, 3)
    s = Stream(w)
    f = make_factored(w, s.V0)
    W = s.V0.astype(np.float64)
    for t in range(24):
        H, idx, val = s.batch()
        if t % 3:
            H, idx, val = H[:1].copy(), idx[:1].copy(), val[:1].copy()
        ref = oracle_step(W, H, idx, val, w)
        loss, g = f.step(*to_dev(H, idx, val), w.lr)
        assert f.sync_status() == 0
        assert abs(loss.item() - ref.loss) <= TOL100 * abs(ref.loss)
        W = ref.W_new
    assert rel(f.materialize_W().cpu().numpy(), W) <= TOL100
    f.close()


def test_online_duplicates_empty_slots_and_untouched_rows():
    w = Workload("t", LOSS_SQUARED, 50, 24, 1, 4, index_dist="zipf")
    s = Stream(w)
    f = make_factored(w, s.V0)
    W = s.V0.astype(np.float64)
    for t in range(12):
        H, idx, val = s.batch()
        idx[0, 1] = idx[0, 0]
        if t % 2:
            idx[0, 3] = -1
        V_before = f.V.clone()
        ref = oracle_step(W, H, idx, val, w)
        loss, g = f.step(*to_dev(H, idx, val), w.lr)
        assert f.sync_status() == 0
        assert abs(loss.item() - ref.loss) <= TOL100 * abs(ref.loss)
        touched = torch.zeros(w.D, dtype=torch.bool, device=DEV)
        valid = idx[0][idx[0] >= 0].astype(np.int64)
        touched[torch.from_numpy(valid).to(DEV)] = True
        assert torch.equal(f.V[~touched], V_before[~touched])
        W = ref.W_new
    assert rel(f.materialize_W().cpu().numpy(), W) <= TOL100
    f.close()


def _state(f):
    return [t.clone() for t in (f.V, f.U, f.UinvT, f.Q)]


@pytest.mark.parametrize("case", ["index", "nan", "not_spd"])
def test_online_rejected_step_changes_nothing(case):
    w = Workload("t", LOSS_SQUARED, 300, 16, 1, 2, lr=0.05)
    s = Stream(w)
    f = make_factored(w, s.V0)
    H, idx, val = s.batch()
    want = lst.LST_E_INDEX
    if case == "index":
        idx[0, 1] = w.D
    elif case == "nan":
        H[0, 3] = np.nan
        want = lst.LST_E_NONFINITE
    else:
        H[0] = H[0] / np.linalg.norm(H[0]) * np.sqrt(1.0 / w.lr)  # 1 - 2 eta ||h||^2 = -1
        want = lst.LST_E_NOT_SPD
    snap = _state(f)
    f.step(*to_dev(H.astype(np.float32), idx, val), w.lr)
    assert f.sync_status() == want
    assert all(torch.equal(a, b) for a, b in zip(snap, _state(f)))
    # the context goes on normally afterwards
    H, idx, val = s.batch()
    ref = oracle_step(s.V0.astype(np.float64), H, idx, val, w)
    loss, _ = f.step(*to_dev(H, idx, val), w.lr)
    assert f.sync_status() == 0 and abs(loss.item() - ref.loss) <= TOL1 * abs(ref.loss)
    f.close()

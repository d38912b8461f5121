"""Failure paths of the HIP step, forced from the host with ordinary (in-bounds) inputs.

Every device-detected error must leave V, U, U^{-T} and Q bit-identical to
their values before the failing step, keep later steps from writing until the
host has read the status, and surface as the expected lst_status.  The
expected status is predicted on the CPU (index range, finiteness, and the
Woodbury matrix C = 1 - 2 eta ||h||^2 computed by the factored fp64 mirror).
"""
import numpy as np
import pytest
import torch

import paper_1606_08061_amd as lst
from gpu_common import DEV, make_factored, make_naive, oracle_step, rel, to_dev
from oracle import factored_init
from oracle.factored import alg4_step
from workloads import LOSS_SQUARED, Stream, Workload

pytestmark = pytest.mark.gpu

W_SMALL = Workload("t", LOSS_SQUARED, 1000, 32, 8, 2)


def _state(f):
    return [t.clone() for t in (f.V, f.U, f.UinvT, f.Q)]


def _same(f, snap):
    return all(torch.equal(a, b) for a, b in zip((f.V, f.U, f.UinvT, f.Q), snap))


@pytest.mark.parametrize("bad", [1000, 5000, -2, -7])
def test_index_out_of_range(bad):
    w = W_SMALL
    s = Stream(w)
    f = make_factored(w, s.V0)
    H, idx, val = s.batch()
    f.step(*to_dev(H, idx, val), w.lr)
    assert f.sync_status() == lst.LST_OK
    snap = _state(f)
    H, idx, val = s.batch()
    idx[3, 1] = bad
    assert not (0 <= bad < w.D or bad == -1)  # the oracle side rejects it too
    f.step(*to_dev(H, idx, val), w.lr)
    assert f.sync_status() == lst.LST_E_INDEX
    assert _same(f, snap)
    # the flag was cleared by reading it: a valid step now proceeds and matches the oracle
    W = f.materialize_W().cpu().numpy().astype(np.float64)
    H, idx, val = s.batch()
    loss, g = f.step(*to_dev(H, idx, val), w.lr)
    assert f.sync_status() == lst.LST_OK
    ref = oracle_step(W, H, idx, val, w)
    assert abs(loss.item() - ref.loss) <= 1e-4 * abs(ref.loss)
    assert rel(f.materialize_W().cpu().numpy(), ref.W_new) <= 1e-4
    f.close()


def test_nonfinite_H():
    w = W_SMALL
    s = Stream(w)
    f = make_factored(w, s.V0)
    snap = _state(f)
    H, idx, val = s.batch()
    H[2, 5] = np.nan
    f.step(*to_dev(H, idx, val), w.lr)
    assert f.sync_status() == lst.LST_E_NONFINITE
    assert _same(f, snap)
    f.close()


@pytest.mark.parametrize("m,bad,d", [(1, 0, 16), (70, 40, 16), (200, 150, 16), (300, 290, 16),
                                     (200, 150, 256), (300, 290, 320)])
def test_not_positive_definite(m, bad, d):
    # Example `bad` gets ||h||^2 = 1/eta, so C = I - 2 eta H H^T has C_bad,bad = -1
    # and a negative eigenvalue (for m = 1 this is the Sherman-Morrison denominator
    # 1 - 2 eta ||h||^2 = -1).  With d >= m, elimination of C meets the first
    # non-positive pivot at or before row `bad`, inside a later diagonal block for
    # m > 32; with m > 128 and d < m the branch eliminates the d x d I - 2 eta H^T H,
    # which shares C's negative eigenvalue.  The fp64 mirror confirms C is indefinite.
    w = Workload("t", LOSS_SQUARED, 400, d, m, 1, lr=0.05)
    s = Stream(w)
    H, idx, val = s.batch()
    H = (H * 0.05).astype(np.float32)
    H[bad] = (H[bad] / np.linalg.norm(H[bad]) * np.sqrt(1.0 / w.lr)).astype(np.float32)
    st = factored_init(s.V0)
    _, _, inter = alg4_step(st, H, idx, val, np.float32(w.lr), LOSS_SQUARED)
    assert np.linalg.eigvalsh(inter["C"]).min() < 0
    f = make_factored(w, s.V0)
    snap = _state(f)
    f.step(*to_dev(H, idx, val), w.lr)
    assert f.sync_status() == lst.LST_E_NOT_SPD
    assert _same(f, snap)
    f.close()


def test_error_is_sticky_until_read():
    w = W_SMALL
    s = Stream(w)
    f = make_factored(w, s.V0)
    snap = _state(f)
    H, idx, val = s.batch()
    idx[0, 0] = w.D + 3
    f.step(*to_dev(H, idx, val), w.lr)
    for _ in range(3):  # valid steps enqueued before the host reads the status: no writes
        f.step(*to_dev(*s.batch()), w.lr)
    assert f.sync_status() == lst.LST_E_INDEX
    assert _same(f, snap)
    f.step(*to_dev(*s.batch()), w.lr)
    assert f.sync_status() == lst.LST_OK
    assert not _same(f, snap)
    f.close()


def test_host_argument_errors_enqueue_nothing():
    w = W_SMALL
    s = Stream(w)
    f = make_factored(w, s.V0)
    snap = _state(f)
    H, idx, val = to_dev(*s.batch())
    big = Workload("t", LOSS_SQUARED, 1000, 32, 9, 2)
    Hb, ib, vb = to_dev(*Stream(big).batch())
    loss = torch.zeros((), device=DEV)
    P = lambda t: t.data_ptr()  # noqa: E731
    assert lst.lst_step(f.ctx, P(Hb), 9, P(ib), P(vb), 2, 0.01, P(loss), 0) == lst.LST_E_SHAPE
    assert lst.lst_step(f.ctx, P(H), 8, P(idx), P(val), 3, 0.01, P(loss), 0) == lst.LST_E_SHAPE
    for lr in (0.0, -0.1, float("nan"), float("inf")):
        assert lst.lst_step(f.ctx, P(H), 8, P(idx), P(val), 2, lr, P(loss), 0) == lst.LST_E_ARG
    assert lst.lst_step(f.ctx, 0, 8, P(idx), P(val), 2, 0.01, P(loss), 0) == lst.LST_E_ARG
    assert lst.lst_step(f.ctx, P(H), 8, P(idx), P(val), 2, 0.01, 0, 0) == lst.LST_E_ARG
    assert lst.lst_naive_step(f.ctx, P(H), 8, P(idx), P(val), 2, 0.01, P(loss), 0) == \
        lst.LST_E_STATE
    assert f.sync_status() == lst.LST_OK
    assert _same(f, snap)
    f.close()


def test_naive_index_error_keeps_W():
    w = W_SMALL
    s = Stream(w)
    n = make_naive(w, s.V0)
    W0 = n.W.clone()
    H, idx, val = s.batch()
    idx[1, 0] = w.D
    n.step(*to_dev(H, idx, val), w.lr)
    assert n.sync_status() == lst.LST_E_INDEX
    assert torch.equal(n.W, W0)
    n.close()


def test_online_barrier_expiry_is_all_or_nothing():
    """The one-launch online step (m = 1) meets at a bounded grid barrier.  With its
    spin limit set to 0 (LST_OPT_SPIN_LIMIT) every waiting workgroup gives up at once:
    the single go/abort decision must be abort, so no workgroup writes its part of the
    state (V, U, U^{-T}, Q bit-identical) and the step reports LST_E_SYNC; every kernel
    still finishes (the wait, not the GPU, gives up).  With the limit restored the next
    step matches the oracle."""
    w = Workload("t", LOSS_SQUARED, 2000, 64, 1, 3)
    s = Stream(w)
    f = make_factored(w, s.V0)
    f.set_option(lst.LST_OPT_SPIN_LIMIT, 0)
    snap = _state(f)
    H, idx, val = s.batch()
    f.profile(True)
    f.step(*to_dev(H, idx, val), w.lr)
    assert f.sync_status() == lst.LST_E_SYNC
    assert f.profile_read()["online"][0] == 1  # the one-launch kernel ran
    f.profile(False)
    assert _same(f, snap)
    f.set_option(lst.LST_OPT_SPIN_LIMIT, 1 << 20)
    ref = oracle_step(s.V0.astype(np.float64), H, idx, val, w)
    loss, grad = f.step(*to_dev(H, idx, val), w.lr)
    assert f.sync_status() == lst.LST_OK
    assert abs(loss.item() - ref.loss) <= 1e-4 * abs(ref.loss)
    assert rel(f.materialize_W().cpu().numpy(), ref.W_new) <= 1e-4
    f.close()

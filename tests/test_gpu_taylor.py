"""The Taylor softmax on the GPU: the factored step with dl/ds (omega, w_bar and the
grad_s terms of Z^ and M) and the naive step against the fp64 oracle, the state's
w_bar = W^T 1_D and Q = W^T W, an initial omega, the section 5 restore, and a failing
step that leaves every state array (WO included) bit-identical."""
import numpy as np
import pytest
import torch

import paper_1606_08061_amd as lst
from gpu_common import DEV, Compare, make_factored, oracle_step, rel, to_dev
from workloads import LOSS_TAYLOR_SOFTMAX, Stream, Workload

pytestmark = pytest.mark.gpu

TOL1 = 1e-4
TOL100 = 1e-3


def _wbar_q_ok(f, W, tol):
    W = np.asarray(W, dtype=np.float64)
    assert rel(f.wbar.cpu().numpy(), W.sum(axis=0)) <= tol
    assert rel(f.Q.cpu().numpy(), W.T @ W) <= tol


def _check(st, l, g, ref, tol):
    assert st == 0
    assert abs(l - ref.loss) <= tol * abs(ref.loss), (l, ref.loss)
    assert rel(g, ref.grad_H) <= tol


@pytest.mark.parametrize("D,d,m,K,dist", [
    (5000, 48, 32, 1, "zipf"), (3000, 72, 40, 3, "zipf"), (2000, 33, 17, 4, "uniform"),
    (20000, 130, 150, 2, "uniform"),
])
def test_taylor_steps_match_oracle(D, d, m, K, dist):
    # several 16 x 16 tiles with ragged edges, K above and below a wavefront's slot count,
    # m above 128; 20 steps so that omega and w_bar move away from their initial values
    w = Workload("t", LOSS_TAYLOR_SOFTMAX, D, d, m, K, index_dist=dist, value_dist="ones",
                 lr=0.05)
    c = Compare(w, seed=D + d)
    for t in range(20):
        st, l, g, ref = c.step()
        _check(st, l, g, ref, TOL1 if t == 0 else TOL100)
    W = c.W_gpu()
    assert rel(W, c.W) <= TOL100
    assert np.abs(c.ctx.omega.cpu().numpy()).max() > 0
    _wbar_q_ok(c.ctx, c.W, TOL100)
    c.close()


def test_taylor_first_step_state():
    # one step from a fresh state: every bookkeeping array against its definition at 1e-4
    w = Workload("t", LOSS_TAYLOR_SOFTMAX, 4000, 64, 48, 2, index_dist="zipf",
                 value_dist="ones", lr=0.05)
    c = Compare(w)
    st, l, g, ref = c.step()
    _check(st, l, g, ref, TOL1)
    assert rel(c.W_gpu(), ref.W_new) <= TOL1
    _wbar_q_ok(c.ctx, ref.W_new, TOL1)
    U = c.ctx.U.double().cpu().numpy()
    assert np.abs(U @ c.ctx.UinvT.double().cpu().numpy().T - np.eye(w.d)).max() <= 1e-5
    c.close()


def test_taylor_init_with_U0_and_omega():
    # W = V0 U0 + 1 omega0^T: lst_init_factored takes omega from WO[1] and derives w_bar and Q
    rng = np.random.default_rng(5)
    w = Workload("t", LOSS_TAYLOR_SOFTMAX, 1500, 24, 12, 2, value_dist="ones", lr=0.05)
    s = Stream(w)
    U0 = (np.eye(24) + 0.2 * rng.standard_normal((24, 24))).astype(np.float32)
    om = (0.1 * rng.standard_normal(24)).astype(np.float32)
    f = lst.Factored(w.D, w.d, w.m, w.K, w.loss, device=DEV)
    f.WO[1].copy_(torch.from_numpy(om))
    f.init(to_dev(s.V0)[0], to_dev(U0)[0])
    f.check("init")
    W = s.V0.astype(np.float64) @ U0.astype(np.float64) + om.astype(np.float64)[None, :]
    _wbar_q_ok(f, W, 1e-5)
    assert rel(f.materialize_W().cpu().numpy(), W) <= 1e-6
    for t in range(5):
        H, idx, val = s.batch()
        ref = oracle_step(W, H, idx, val, w)
        loss, g = f.step(*to_dev(H, idx, val), w.lr)
        _check(f.sync_status(), loss.item(), g.cpu().numpy(), ref, TOL1 if t == 0 else TOL100)
        W = ref.W_new
    assert rel(f.materialize_W().cpu().numpy(), W) <= TOL100
    f.close()


def test_taylor_restore_pristine_keeps_W():
    w = Workload("t", LOSS_TAYLOR_SOFTMAX, 3000, 40, 16, 2, index_dist="zipf",
                 value_dist="ones", lr=0.05)
    c = Compare(w)
    for _ in range(5):
        assert c.step()[0] == 0
    W0 = c.W_gpu()
    om = c.ctx.omega.clone()
    c.ctx.restore_pristine()
    c.ctx.check("restore")
    assert torch.equal(om, c.ctx.omega)
    assert rel(c.W_gpu(), W0) <= 1e-6
    st, l, g, ref = c.step()
    _check(st, l, g, ref, TOL100)
    assert rel(c.W_gpu(), c.W) <= TOL100
    c.close()


def test_taylor_failed_step_changes_nothing():
    w = Workload("t", LOSS_TAYLOR_SOFTMAX, 1000, 32, 8, 2, value_dist="ones", lr=0.05)
    s = Stream(w)
    f = make_factored(w, s.V0)
    f.step(*to_dev(*s.batch()), w.lr)
    assert f.sync_status() == lst.LST_OK
    snap = [t.clone() for t in (f.V, f.U, f.UinvT, f.Q, f.WO)]
    H, idx, val = s.batch()
    idx[2, 1] = w.D
    f.step(*to_dev(H, idx, val), w.lr)
    assert f.sync_status() == lst.LST_E_INDEX
    assert all(torch.equal(a, b) for a, b in zip((f.V, f.U, f.UinvT, f.Q, f.WO), snap))
    f.close()


def test_taylor_naive_matches_oracle_and_factored():
    # the naive path: column sums of O for s, 1 ds^T in grad_O; m = 20 takes the 128 x 128-tile
    # forward product, m = 13 (d = 30) the general one
    for D, d, m, K in ((3000, 40, 20, 1), (2500, 30, 13, 2)):
        w = Workload("t", LOSS_TAYLOR_SOFTMAX, D, d, m, K, index_dist="zipf", value_dist="ones",
                     lr=0.05)
        c = Compare(w, path="naive")
        for t in range(10):
            st, l, g, ref = c.step()
            _check(st, l, g, ref, TOL1 if t == 0 else TOL100)
        assert rel(c.W_gpu(), c.W) <= TOL100
        c.close()
    w = Workload("t", LOSS_TAYLOR_SOFTMAX, 4000, 64, 32, 2, index_dist="zipf",
                 value_dist="ones", lr=0.05)
    s = Stream(w)
    f = make_factored(w, s.V0)
    n = lst.Naive(w.D, w.d, w.m, w.K, w.loss, device=DEV)
    n.init(to_dev(s.V0)[0])
    for _ in range(20):
        b = to_dev(*s.batch())
        lf, _ = f.step(*b, w.lr)
        ln, _ = n.step(*b, w.lr)
        assert abs(lf.item() - ln.item()) <= 1e-3 * abs(ln.item())
    f.check()
    n.check()
    assert rel(f.materialize_W().cpu().numpy(), n.W.cpu().numpy()) <= 1e-3
    f.close()
    n.close()

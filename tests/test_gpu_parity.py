"""Parity of the HIP path (through the C ABI) with the fp64 dense oracle.

Tolerances: relative error <= 1e-4 on the loss and on grad_H (Frobenius) for a
single step; <= 1e-3 on V U after 100 steps; integer/index results bit exact
(rows of V outside a step's targets are unchanged bit for bit).
"""
import numpy as np
import pytest
import torch

from gpu_common import DEV, Compare, make_factored, oracle_step, rel, to_dev
from oracle import dense_step
from workloads import (LOSS_SPHERICAL_SOFTMAX, LOSS_SQUARED, LOSS_TAYLOR_SOFTMAX, WORKLOADS,
                       Stream, Workload)

pytestmark = pytest.mark.gpu

TOL1 = 1e-4
TOL100 = 1e-3


def _check_step(st, loss, grad, ref, tol=TOL1):
    assert st == 0
    assert abs(loss - ref.loss) <= tol * abs(ref.loss), (loss, ref.loss)
    assert rel(grad, ref.grad_H) <= tol


def test_small_config_single_step_and_invariants():
    w = WORKLOADS["sq_D2k_d32_m16_K3"]
    c = Compare(w)
    st, loss, grad, ref = c.step()
    _check_step(st, loss, grad, ref)
    Wg = c.W_gpu()
    assert rel(Wg, ref.W_new) <= TOL1
    f = c.ctx
    Q = f.Q.cpu().numpy().astype(np.float64)
    U = f.U.cpu().numpy().astype(np.float64)
    UinvT = f.UinvT.cpu().numpy().astype(np.float64)
    assert rel(Q, ref.W_new.T @ ref.W_new) <= TOL1
    assert np.abs(U @ UinvT.T - np.eye(w.d)).max() <= 1e-5
    c.close()


def test_small_config_100_steps():
    w = WORKLOADS["sq_D2k_d32_m16_K3"]
    c = Compare(w)
    for t in range(w.steps):
        st, loss, grad, ref = c.step()
        _check_step(st, loss, grad, ref, TOL1 if t == 0 else TOL100)
    assert rel(c.W_gpu(), c.W) <= TOL100
    c.close()


@pytest.mark.parametrize("loss", [LOSS_SQUARED, LOSS_SPHERICAL_SOFTMAX, LOSS_TAYLOR_SOFTMAX])
@pytest.mark.parametrize("D,d,m,K", [
    (50, 1, 1, 1), (300, 31, 2, 3), (1000, 33, 17, 2), (777, 65, 33, 1), (2000, 40, 70, 3),
    (1500, 47, 130, 2), (3000, 24, 300, 1), (2500, 20, 520, 1), (400, 64, 5, 0),
    # m above 128, with d above and below m (E = 2 eta S H H^T S of rank min(m, d))
    (2000, 160, 150, 2), (1200, 300, 260, 1), (1800, 200, 260, 2),
])
def test_awkward_shapes(loss, D, d, m, K):
    w = Workload("t", loss, D, d, m, K, index_dist="uniform",
                 value_dist="normal" if loss == LOSS_SQUARED else "ones", lr=0.01)
    c = Compare(w, seed=D + d + m + K)
    for t in range(4):
        st, l, g, ref = c.step()
        _check_step(st, l, g, ref, TOL1 if t == 0 else TOL100)
    assert rel(c.W_gpu(), c.W) <= TOL100
    c.close()


def test_spherical_softmax_zipf_steps():
    w = Workload("t", LOSS_SPHERICAL_SOFTMAX, 5000, 48, 32, 1, index_dist="zipf",
                 value_dist="ones", steps=30)
    c = Compare(w)
    for t in range(w.steps):
        st, l, g, ref = c.step()
        _check_step(st, l, g, ref, TOL1 if t == 0 else TOL100)
    assert rel(c.W_gpu(), c.W) <= TOL100
    c.close()


def _dup_batch(c, t):
    H, idx, val = c.s.batch()
    idx[0, 1] = idx[0, 0]
    idx[1, 2] = -1
    if t % 3 == 0:
        idx[2, :] = -1
    return H, idx, val


@pytest.mark.parametrize("loss,D,K", [
    (LOSS_SQUARED, 9, 3), (LOSS_SPHERICAL_SOFTMAX, 9, 3), (LOSS_SQUARED, 40, 16),
    (LOSS_SQUARED, 60, 20), (LOSS_TAYLOR_SOFTMAX, 9, 3), (LOSS_TAYLOR_SOFTMAX, 40, 16),
])
def test_duplicates_and_empty_slots(loss, D, K):
    # small D under Zipf: rows repeat across examples; some examples repeat an index or have
    # -1; Yring^T Yring from the merged slot lists (K = 20: two 16-entry chunks).
    w = Workload("t", loss, D, 8, 24, K, index_dist="zipf",
                 value_dist="normal" if loss == LOSS_SQUARED else "ones")
    c = Compare(w)
    for t in range(10):
        st, l, g, ref = c.step(_dup_batch(c, t))
        _check_step(st, l, g, ref, TOL1 if t == 0 else TOL100)
    assert rel(c.W_gpu(), c.W) <= TOL100
    c.close()


@pytest.mark.parametrize("loss,D,d,m,K", [
    (LOSS_SQUARED, 8, 40, 128, 8), (LOSS_SQUARED, 3, 37, 96, 3), (LOSS_SQUARED, 48, 24, 120, 48),
    (LOSS_SPHERICAL_SOFTMAX, 3, 40, 128, 1), (LOSS_TAYLOR_SOFTMAX, 3, 40, 128, 1),
    (LOSS_SQUARED, 8, 32, 1024, 8),  # m K = 8192, the largest: 32 chunks a row
])
def test_frequent_rows_summed_in_chunks(loss, D, d, m, K):
    # A V row with more than max(32, K) slots is summed by several workgroups (chunks of
    # that many slots, partial sums added in chunk order by the last to arrive): with D <= K
    # every example targets every row, so each row has m slots (3 or 4 chunks); d = 37 takes
    # the one-column partial sums, K = 48 the chunk size K; the softmax losses (one-hot
    # targets over D = 3 classes, about 43 slots a row: two chunks) weight the slots by
    # their own dl/dA.
    w = Workload("t", loss, D, d, m, K, index_dist="uniform", lr=1e-3,
                 value_dist="normal" if loss == LOSS_SQUARED else "ones")
    c = Compare(w, seed=D * 1000 + K)
    for t in range(5):
        st, l, g, ref = c.step()
        _check_step(st, l, g, ref, TOL1 if t == 0 else TOL100)
    assert rel(c.W_gpu(), c.W) <= TOL100
    c.close()


def test_duplicates_spherical_softmax_most_classes_targeted():
    # The spherical softmax with K = 16 slots over D = 40 classes (Zipf), the same repeated
    # and empty slots.  With most classes targeted many a_kj sit near 0, where d/da of
    # a / (a^2 + eps) is 1 / eps, and this workload's trajectory magnifies any rounding
    # difference about fourfold per step: the dense definition itself, run in fp32 along its
    # own trajectory, is 3.5e-3 away from the fp64 one after ten steps.  Parity is therefore
    # taken one step at a time from the GPU's own state: the oracle steps W = V U formed in
    # fp64 from the context's fp32 V and U, and the step's loss, grad_H and updated V U must
    # match it to 1e-4 (the fp32 definition is within 1e-6 of it from the same state).
    w = Workload("t", LOSS_SPHERICAL_SOFTMAX, 40, 8, 24, 16, index_dist="zipf",
                 value_dist="ones")
    c = Compare(w)

    def W_exact():
        return c.ctx.V.double().cpu().numpy() @ c.ctx.U.double().cpu().numpy()

    for t in range(30):
        H, idx, val = _dup_batch(c, t)
        ref = oracle_step(W_exact(), H, idx, val, w)
        loss, grad = c.ctx.step(*to_dev(H, idx, val), w.lr)
        assert c.ctx.sync_status() == 0
        assert abs(loss.item() - ref.loss) <= TOL1 * abs(ref.loss), t
        assert rel(grad.cpu().numpy(), ref.grad_H) <= TOL1, t
        assert rel(W_exact(), ref.W_new) <= TOL1, t
    c.close()


@pytest.mark.parametrize("loss,d", [(LOSS_SQUARED, 512), (LOSS_SQUARED, 1024),
                                    (LOSS_SQUARED, 700), (LOSS_SPHERICAL_SOFTMAX, 700),
                                    (LOSS_TAYLOR_SOFTMAX, 700)])
def test_sweep_minibatch_m512(loss, d):
    # the sweep's m = 512 (32 tile rows of every m x m product of the Woodbury polynomial;
    # 512 < d <= 1024 takes the gather with 16 columns per lane; d = 700 is no multiple of
    # 64), at D = 20000: the whole updated W after one step, and a second step.
    K = 5 if loss == LOSS_SQUARED else 1
    w = Workload("t", loss, 20000, d, 512, K,
                 value_dist="normal" if loss == LOSS_SQUARED else "ones")
    c = Compare(w, seed=d)
    st, l, g, ref = c.step()
    _check_step(st, l, g, ref)
    assert rel(c.W_gpu(), ref.W_new) <= TOL1
    st, l, g, ref = c.step()
    _check_step(st, l, g, ref, TOL100)
    assert rel(c.W_gpu(), c.W) <= TOL100
    c.close()


@pytest.mark.parametrize("loss,d,m", [(LOSS_SQUARED, 514, 458), (LOSS_SPHERICAL_SOFTMAX, 516, 460),
                                      (LOSS_TAYLOR_SOFTMAX, 514, 458), (LOSS_SQUARED, 1022, 258),
                                      (LOSS_SQUARED, 1000, 300)])
def test_large_ragged_shapes_on_64_tiles(loss, d, m):
    # shapes large enough for the LDS-staged 64 x 64 tiles, with ragged tile edges: m near
    # 512 puts launches 1 and 3 on them, d near 1024 launches 4 and 5 (with Zq's and R X's
    # operand terms); d = 514 or 1022 and m = 258 or 458 are no multiples of 4 (the scalar
    # operand loads)
    K = 3 if loss == LOSS_SQUARED else 1
    w = Workload("t", loss, 20000, d, m, K,
                 value_dist="normal" if loss == LOSS_SQUARED else "ones")
    c = Compare(w, seed=d + m)
    st, l, g, ref = c.step()
    _check_step(st, l, g, ref)
    assert rel(c.W_gpu(), ref.W_new) <= TOL1
    st, l, g, ref = c.step()
    _check_step(st, l, g, ref, TOL100)
    assert rel(c.W_gpu(), c.W) <= TOL100
    c.close()


def _poly_bound(H, dq, lr):
    """||E^2||_inf^(1/2) of E = 2 lr S H H^T S (S = diag(dq)^(1/2)), in fp64: the bound on the
    spectral radius the step's certificate takes."""
    Hs = np.sqrt(dq)[:, None] * H.astype(np.float64)
    E = 2.0 * float(lr) * (Hs @ Hs.T)
    return float(np.sqrt(np.abs(E @ E).sum(1).max()))


@pytest.mark.parametrize("m,d", [(64, 32), (200, 48), (512, 1024)])
def test_uncertified_woodbury_takes_exact_elimination(m, d):
    # Steps large enough (2 eta lambda_max(H H^T) = 0.6) that the degree-7 polynomial cannot
    # certify C^{-1} = (I - 2 eta H H^T)^{-1} (its bound needs ||E^2||^(1/2) <= 0.3), while C is
    # still positive definite: one workgroup inverts C by exact elimination (m = 200: beyond
    # the 128 rows the tiles of one product hold; m = 512, d = 1024: R X on 64 x 64 tiles
    # takes its alternative), and the step matches the oracle.
    w = Workload("t", LOSS_SQUARED, 3000, d, m, 3)
    s = Stream(w, seed=m)
    f = make_factored(w, s.V0)
    W = s.V0.astype(np.float64)
    for t in range(3):
        H, idx, val = s.batch()
        lam = float(np.linalg.eigvalsh(H.astype(np.float64) @ H.astype(np.float64).T).max())
        lr = float(np.float32(0.3 / lam))
        assert _poly_bound(H, np.ones(m), lr) > 0.31  # not certifiable
        ref = dense_step(W, H, idx, val, np.float32(lr), w.loss)
        loss, grad = f.step(*to_dev(H, idx, val), lr)
        st = f.sync_status()
        _check_step(st, loss.item(), grad.cpu().numpy(), ref, TOL1 if t == 0 else TOL100)
        W = ref.W_new
    assert rel(f.materialize_W().cpu().numpy(), W) <= TOL100
    f.close()


def test_all_slots_same_row():
    w = Workload("t", LOSS_SQUARED, 100, 16, 40, 4)
    c = Compare(w)
    for _ in range(3):
        H, idx, val = c.s.batch()
        idx[:, :] = 7
        st, l, g, ref = c.step((H, idx, val))
        _check_step(st, l, g, ref, 1e-3)
    assert rel(c.W_gpu(), c.W) <= TOL100
    c.close()


def test_general_U0():
    rng = np.random.default_rng(3)
    w = Workload("t", LOSS_SQUARED, 1200, 24, 10, 2)
    U0 = (np.eye(24) + 0.2 * rng.standard_normal((24, 24))).astype(np.float32)
    c = Compare(w, U0=U0)
    for t in range(5):
        st, l, g, ref = c.step()
        _check_step(st, l, g, ref, 1e-4 if t == 0 else 1e-3)
    assert rel(c.W_gpu(), c.W) <= 1e-3
    c.close()


def test_naive_path_matches_oracle():
    # the first two run the 128 x 128-tile products (split over D for grad_H, with a
    # ragged last split); m = 13, d = 30 takes the general GEMM and column-norm kernels
    for w in (WORKLOADS["sq_D2k_d32_m16_K3"],
              Workload("t", LOSS_SPHERICAL_SOFTMAX, 3000, 40, 20, 1, index_dist="zipf",
                       value_dist="ones"),
              Workload("t", LOSS_SQUARED, 2500, 30, 13, 2)):
        c = Compare(w, path="naive")
        for t in range(10):
            st, l, g, ref = c.step()
            _check_step(st, l, g, ref, TOL1 if t == 0 else TOL100)
        assert rel(c.W_gpu(), c.W) <= TOL100
        c.close()


def test_factored_and_naive_agree_over_steps():
    w = Workload("t", LOSS_SQUARED, 4000, 64, 32, 3)
    s = Stream(w)
    f = make_factored(w, s.V0)
    import paper_1606_08061_amd as lst
    n = lst.Naive(w.D, w.d, w.m, w.K, w.loss, device=DEV)
    n.init(to_dev(s.V0)[0])
    for _ in range(20):
        b = to_dev(*s.batch())
        lf, gf = f.step(*b, w.lr)
        ln, gn = n.step(*b, w.lr)
        assert abs(lf.item() - ln.item()) <= 1e-3 * abs(ln.item())
    f.check()
    n.check()
    assert rel(f.materialize_W().cpu().numpy(), n.W.cpu().numpy()) <= 1e-3
    f.close()
    n.close()


def test_zero_batch_and_no_targets():
    w = Workload("t", LOSS_SQUARED, 500, 16, 8, 2)
    c = Compare(w)
    V = c.ctx.V.clone()
    H, idx, val = c.s.batch()
    loss, _ = c.ctx.step(*to_dev(H[:0], idx[:0], val[:0]), w.lr)
    assert c.ctx.sync_status() == 0 and loss.item() == 0.0
    assert torch.equal(V, c.ctx.V)
    # K = 0: no targets, y = 0
    st, l, g, ref = c.step((H, idx[:, :0].copy(), val[:, :0].copy()))
    _check_step(st, l, g, ref)
    c.close()


@pytest.mark.parametrize("d,m", [(96, 64), (1024, 512)])
def test_untouched_rows_bit_identical_and_deterministic(d, m):
    # (d = 1024, m = 512: every launch's products on the 64 x 64 tiles, Zq's and R X's
    # operand terms included)
    w = Workload("t", LOSS_SQUARED, 20000, d, m, 4, index_dist="zipf")
    s = Stream(w)
    batches = [s.batch() for _ in range(5)]
    outs = []
    for rep in range(2):
        f = make_factored(w, s.V0)
        for H, idx, val in batches:
            V_before = f.V.clone()
            loss, g = f.step(*to_dev(H, idx, val), w.lr)
            f.check()
            touched = torch.zeros(w.D, dtype=torch.bool, device=DEV)
            touched[torch.from_numpy(idx.reshape(-1).astype(np.int64)).to(DEV)] = True
            assert torch.equal(f.V[~touched], V_before[~touched])
            assert not torch.equal(f.V[touched], V_before[touched])
        outs.append([t.clone() for t in (f.V, f.U, f.UinvT, f.Q, loss, g)])
        f.close()
    for a, b in zip(*outs):
        assert torch.equal(a, b)


@pytest.mark.parametrize("loss", [LOSS_SQUARED, LOSS_SPHERICAL_SOFTMAX, LOSS_TAYLOR_SOFTMAX])
def test_graph_replay_matches_eager(loss):
    # Each step's arguments recur every third step, so the cached graphs are replayed several
    # times, with eager torch work and host synchronisations between the replays; every replay
    # must give bit-identical results to kernel-by-kernel enqueueing.
    w = Workload("t", loss, 5000, 64, 32, 3, value_dist="normal" if loss == LOSS_SQUARED else "ones")
    s = Stream(w)
    batches = [to_dev(*s.batch()) for _ in range(3)]
    outs = []
    for graphs in (False, True):
        f = make_factored(w, s.V0)
        f.use_graphs(graphs)
        loss_buf = torch.zeros((), device=DEV)
        grad_buf = torch.empty((w.m, w.d), device=DEV)
        losses, grads = [], []
        for t in range(9):
            f.step(*batches[t % 3], w.lr, grad_H=grad_buf, loss_out=loss_buf)
            losses.append(loss_buf.item())
            grads.append(grad_buf.clone())
            assert torch.ones(7, device=DEV).sum().item() == 7.0
        f.check()
        outs.append((losses, grads, [t.clone() for t in (f.V, f.U, f.UinvT, f.Q)]))
        f.close()
    (l0, g0, s0), (l1, g1, s1) = outs
    assert l0 == l1
    for a, b in zip(g0, g1):
        assert torch.equal(a, b)
    for a, b in zip(s0, s1):
        assert torch.equal(a, b)

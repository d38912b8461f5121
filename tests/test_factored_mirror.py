"""The paper's factored algebra (fp64 mirror of Algorithms 3 and 4) against the dense oracle.

The proofs of sections 3.2, 3.4, 3.6 and 4.4 state that the factored updates
reproduce the dense gradient step exactly; in fp64 the two must agree to
rounding.  Also checked: the invariants Q = W^T W and U (U^{-T})^T = I, the
derived Woodbury form against Sherman-Morrison (eq. updateU-T) at m = 1 and
against a from-scratch inverse, and Algorithm 3 against Algorithm 4 for squared
error (Algorithm 4's M is 4x Algorithm 3's M).
"""
import numpy as np
import pytest

from oracle import dense_step, factored_init
from oracle.factored import alg3_step, alg4_step
from workloads import (LOSS_SPHERICAL_SOFTMAX, LOSS_SQUARED, LOSS_TAYLOR_SOFTMAX, WORKLOADS,
                       Stream, Workload)


def _rel(a, b):
    return np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300)


@pytest.mark.parametrize("alg", ["alg3", "alg4"])
def test_squared_100_steps_match_dense(alg):
    w = WORKLOADS["sq_D2k_d32_m16_K3"]
    s = Stream(w)
    st = factored_init(s.V0)
    W = s.V0.astype(np.float64)
    for t in range(w.steps):
        H, idx, val = s.batch()
        ref = dense_step(W, H, idx, val, w.lr, LOSS_SQUARED)
        if alg == "alg3":
            L, g, _ = alg3_step(st, H, idx, val, w.lr)
        else:
            L, g, _ = alg4_step(st, H, idx, val, w.lr, LOSS_SQUARED)
        W = ref.W_new
        assert L == pytest.approx(ref.loss, rel=1e-10)
        assert _rel(g, ref.grad_H) < 1e-10
        if t % 10 == 9:
            assert _rel(st.W(), W) < 1e-10
            assert _rel(st.Q, W.T @ W) < 1e-10
            assert np.abs(st.U @ st.UinvT.T - np.eye(w.d)).max() < 1e-10
    assert _rel(st.W(), W) < 1e-10


def test_spherical_softmax_steps_match_dense():
    w = Workload("t", LOSS_SPHERICAL_SOFTMAX, 500, 16, 8, 1, index_dist="zipf",
                 value_dist="ones", steps=40)
    s = Stream(w)
    st = factored_init(s.V0)
    W = s.V0.astype(np.float64)
    for _ in range(w.steps):
        H, idx, val = s.batch()
        ref = dense_step(W, H, idx, val, w.lr, LOSS_SPHERICAL_SOFTMAX, w.eps)
        L, g, _ = alg4_step(st, H, idx, val, w.lr, LOSS_SPHERICAL_SOFTMAX, w.eps)
        W = ref.W_new
        assert L == pytest.approx(ref.loss, rel=1e-10)
        assert _rel(g, ref.grad_H) < 1e-10
    assert _rel(st.W(), W) < 1e-10
    assert _rel(st.Q, W.T @ W) < 1e-10


@pytest.mark.parametrize("K,index_dist", [(1, "zipf"), (4, "uniform")])
def test_taylor_softmax_steps_match_dense(K, index_dist):
    # every row of Algorithm 4: s, h~, grad_s, y_bar, the omega and w_bar updates and the
    # grad_s terms of Z^ and M; omega leaves 0 after the first step and w_bar tracks W^T 1
    w = Workload("t", LOSS_TAYLOR_SOFTMAX, 300, 12, 8, K, index_dist=index_dist,
                 value_dist="ones", lr=0.05, steps=30)
    s = Stream(w)
    st = factored_init(s.V0)
    W = s.V0.astype(np.float64)
    assert _rel(st.wbar, W.sum(axis=0)) < 1e-14 and not st.omega.any()
    for _ in range(w.steps):
        H, idx, val = s.batch()
        ref = dense_step(W, H, idx, val, w.lr, LOSS_TAYLOR_SOFTMAX)
        L, g, inter = alg4_step(st, H, idx, val, w.lr, LOSS_TAYLOR_SOFTMAX)
        W = ref.W_new
        assert L == pytest.approx(ref.loss, rel=1e-10)
        assert _rel(g, ref.grad_H) < 1e-10
        assert np.all(inter["ds"] > 0)
    assert np.abs(st.omega).max() > 1e-3
    assert _rel(st.W(), W) < 1e-10
    assert _rel(st.Q, W.T @ W) < 1e-10
    assert _rel(st.wbar, W.sum(axis=0)) < 1e-10
    assert np.abs(st.U @ st.UinvT.T - np.eye(w.d)).max() < 1e-10


@pytest.mark.parametrize("loss", [LOSS_SQUARED, LOSS_SPHERICAL_SOFTMAX, LOSS_TAYLOR_SOFTMAX])
def test_duplicates_across_and_within_examples(loss):
    # Zipf over a tiny D makes many rows repeat across examples; one example repeats an index.
    w = Workload("t", loss, 7, 5, 6, 3, index_dist="zipf",
                 value_dist="normal" if loss == LOSS_SQUARED else "ones")
    s = Stream(w)
    st = factored_init(s.V0)
    W = s.V0.astype(np.float64)
    for t in range(12):
        H, idx, val = s.batch()
        if t % 3 == 0:
            idx[0, 1] = idx[0, 0]
        if t % 4 == 1:
            idx[1, 2] = -1
        ref = dense_step(W, H, idx, val, w.lr, loss, w.eps)
        L, g, _ = alg4_step(st, H, idx, val, w.lr, loss, w.eps)
        W = ref.W_new
        assert L == pytest.approx(ref.loss, rel=1e-10)
        assert _rel(g, ref.grad_H) < 1e-10
    assert _rel(st.W(), W) < 1e-10
    assert _rel(st.Q, W.T @ W) < 1e-10


def test_woodbury_is_sherman_morrison_at_m1():
    rng = np.random.default_rng(0)
    D, d, lr = 30, 6, 0.2
    st = factored_init(rng.standard_normal((D, d)), np.eye(d) + 0.1 * rng.standard_normal((d, d)))
    h = rng.standard_normal((1, d))
    UinvT0 = st.UinvT.copy()
    alg4_step(st, h, np.array([[3]]), np.array([[0.7]]), lr, LOSS_SQUARED)
    hv = h[0]
    sm = UinvT0 + (2 * lr / (1 - 2 * lr * hv @ hv)) * np.outer(UinvT0 @ hv, hv)
    np.testing.assert_allclose(st.UinvT, sm, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(st.UinvT, np.linalg.inv(st.U).T, rtol=1e-10, atol=1e-12)


def test_alg3_equals_alg4_for_squared_error():
    w = Workload("t", LOSS_SQUARED, 300, 12, 9, 4, steps=5)
    s = Stream(w)
    a = factored_init(s.V0)
    b = a.copy()
    for _ in range(w.steps):
        H, idx, val = s.batch()
        L3, g3, i3 = alg3_step(a, H, idx, val, w.lr)
        L4, g4, i4 = alg4_step(b, H, idx, val, w.lr, LOSS_SQUARED)
        assert L3 == pytest.approx(L4, rel=1e-12)
        np.testing.assert_allclose(g3, g4, rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(i4["M"], 4 * i3["M"], rtol=1e-10, atol=1e-10)
    for x, y in ((a.V, b.V), (a.U, b.U), (a.UinvT, b.UinvT), (a.Q, b.Q)):
        assert _rel(x, y) < 1e-11


def test_general_U0():
    rng = np.random.default_rng(4)
    D, d = 50, 7
    V0 = rng.standard_normal((D, d)) / np.sqrt(d)
    U0 = np.eye(d) + 0.3 * rng.standard_normal((d, d))
    st = factored_init(V0, U0)
    W = V0 @ U0
    for _ in range(6):
        H = rng.standard_normal((4, d)) / np.sqrt(d)
        idx = np.stack([rng.choice(D, 2, replace=False) for _ in range(4)])
        val = rng.standard_normal((4, 2))
        ref = dense_step(W, H, idx, val, 0.05, LOSS_SQUARED)
        L, g, _ = alg4_step(st, H, idx, val, 0.05, LOSS_SQUARED)
        W = ref.W_new
        assert L == pytest.approx(ref.loss, rel=1e-10)
    assert _rel(st.W(), W) < 1e-10


def test_not_spd_when_step_too_large():
    # m = 1: C = 1 - 2 eta ||h||^2 (the Sherman-Morrison denominator) vanishes or turns negative
    rng = np.random.default_rng(1)
    h = rng.standard_normal((1, 4))
    lr = 0.75 / (h[0] @ h[0])
    st = factored_init(rng.standard_normal((10, 4)))
    _, _, inter = alg4_step(st, h, np.array([[1]]), np.array([[1.0]]), lr, LOSS_SQUARED)
    assert inter["C"][0, 0] < 0

"""Pins of the section 5 stabilisation oracle against things other than itself.

* LAPACK's SVD (numpy.linalg.svd) for the singular values and left singular
  vectors that the power iteration finds and that fix-singular-value changes;
* the invariant the paper proves for Algorithm 5 and states for section 5.1:
  V U (the implicit W) is unchanged, and so is Q = W^T W;
* the definition of the inverse (U X^T = I) for the recomputed and the
  rank-one-updated U^{-T};
* the method itself: training continues from a restored or stabilised state
  and still matches the dense definition step for step.
"""
import numpy as np
import pytest

from oracle import dense_step, factored_init, factored_step
from oracle.stabilize import (fix_singular_value, largest_singular, power_iteration,
                              reinvert, restore_pristine, singular_stabilize, smallest_singular)


def _orth(rng, d):
    q, r = np.linalg.qr(rng.standard_normal((d, d)))
    return q * np.sign(np.diag(r))


def _state_with_singular_values(seed, D, sig):
    """A factored state whose U has exactly the singular values sig."""
    rng = np.random.default_rng(seed)
    d = len(sig)
    U = _orth(rng, d) @ np.diag(sig) @ _orth(rng, d).T
    return factored_init(rng.standard_normal((D, d)), U), rng


def _same_direction(u, v, tol):
    return abs(abs(np.dot(u, v)) - 1.0) <= tol


def test_restore_keeps_W_and_Q_and_resets_U():
    st, _ = _state_with_singular_values(0, 40, np.linspace(0.3, 3.0, 6))
    W = st.V @ st.U
    r = restore_pristine(st)
    np.testing.assert_allclose(r.V, W, rtol=0, atol=1e-12)
    assert np.array_equal(r.U, np.eye(6)) and np.array_equal(r.UinvT, np.eye(6))
    np.testing.assert_allclose(r.Q, W.T @ W, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("loss", ["squared", "spherical_softmax"])
def test_training_continues_after_restore_and_fix(loss):
    # the stabilised state still represents W: factored steps from it equal dense steps on W
    st, rng = _state_with_singular_values(1, 30, np.array([0.05, 0.7, 1.0, 2.0, 9.0]))
    for op in ("restore", "fix"):
        s = restore_pristine(st) if op == "restore" else None
        if op == "fix":
            u, sig = smallest_singular(st, rng.standard_normal(5), 64)
            s = fix_singular_value(st, sig, u, 1.0)
        W = s.V @ s.U
        for _ in range(3):
            H = rng.standard_normal((4, 5)) / np.sqrt(5)
            idx = rng.integers(0, 30, size=(4, 2)).astype(np.int32)
            val = np.ones((4, 2)) if loss == "spherical_softmax" else rng.standard_normal((4, 2))
            ref = dense_step(W, H, idx, val, 0.05, loss)
            L, g, _ = factored_step(s, H, idx, val, 0.05, loss)
            W = ref.W_new
            assert L == pytest.approx(ref.loss, rel=1e-10)
            np.testing.assert_allclose(g, ref.grad_H, rtol=1e-9, atol=1e-11)
            np.testing.assert_allclose(s.V @ s.U, W, rtol=1e-9, atol=1e-10)


def test_reinvert_is_the_inverse():
    st, _ = _state_with_singular_values(2, 10, np.array([1e-2, 0.5, 1.0, 4.0, 30.0]))
    st.UinvT = st.UinvT + 1e-3  # a drifted carried value must not matter
    r = reinvert(st)
    np.testing.assert_allclose(st.U @ r.UinvT.T, np.eye(5), atol=1e-10)
    np.testing.assert_allclose(r.UinvT.T @ st.U, np.eye(5), atol=1e-10)


def test_power_iteration_matches_svd():
    sig = np.array([0.2, 0.5, 1.0, 1.5, 6.0, 0.9, 3.0])
    st, rng = _state_with_singular_values(3, 12, sig)
    Ub, s, _ = np.linalg.svd(st.U)
    u0 = rng.standard_normal(7)
    u, smax = largest_singular(st, u0, 128)
    assert smax == pytest.approx(s[0], rel=1e-12) and smax == pytest.approx(6.0, rel=1e-12)
    assert _same_direction(u, Ub[:, 0], 1e-12)
    u, smin = smallest_singular(st, u0, 128)
    assert smin == pytest.approx(s[-1], rel=1e-12) and smin == pytest.approx(0.2, rel=1e-12)
    assert _same_direction(u, Ub[:, -1], 1e-12)


def test_power_iteration_diagonal_closed_form():
    # A = diag(a): u converges to the unit vector of the largest |a_i|, sigma = max |a_i|
    a = np.array([0.5, -4.0, 2.0, 1.0])
    u, s = power_iteration(np.diag(a), np.ones(4), 200)
    assert s == pytest.approx(4.0, rel=1e-14)
    assert _same_direction(u, np.array([0.0, 1.0, 0.0, 0.0]), 1e-14)


@pytest.mark.parametrize("which", ["smallest", "largest"])
def test_fix_singular_value(which):
    sig = np.array([0.01, 0.4, 1.0, 2.5, 50.0, 0.8])
    st, rng = _state_with_singular_values(4, 25, sig)
    W = st.V @ st.U
    find = smallest_singular if which == "smallest" else largest_singular
    u, s = find(st, rng.standard_normal(6), 256)
    f = fix_singular_value(st, s, u, 1.0)
    # the paper's proof: W = V U unchanged; Q therefore too
    np.testing.assert_allclose(f.V @ f.U, W, rtol=1e-11, atol=1e-11)
    np.testing.assert_array_equal(f.Q, st.Q)
    # the fixed singular value is 1, the others are unchanged (LAPACK's SVD)
    want = sig.copy()
    want[np.argmin(sig) if which == "smallest" else np.argmax(sig)] = 1.0
    np.testing.assert_allclose(np.sort(np.linalg.svd(f.U, compute_uv=False)), np.sort(want),
                               rtol=1e-10)
    # the rank-one update of U^{-T} is the inverse of the new U
    np.testing.assert_allclose(f.U @ f.UinvT.T, np.eye(6), atol=1e-10)


def test_fix_to_other_targets():
    st, rng = _state_with_singular_values(5, 8, np.array([0.3, 1.0, 2.0]))
    u, s = largest_singular(st, rng.standard_normal(3), 256)
    f = fix_singular_value(st, s, u, 0.5)
    np.testing.assert_allclose(np.sort(np.linalg.svd(f.U, compute_uv=False)), [0.3, 0.5, 1.0],
                               rtol=1e-10)
    np.testing.assert_allclose(f.V @ f.U, st.V @ st.U, rtol=1e-11, atol=1e-11)


def test_singular_stabilize_brings_every_value_into_range():
    sig = np.array([1e-4, 5e-4, 0.02, 0.7, 1.0, 3.0, 80.0, 400.0])
    st, rng = _state_with_singular_values(6, 50, sig)
    W = st.V @ st.U
    out, n_lo, n_hi, s_min, s_max = singular_stabilize(st, rng.standard_normal(8), 128,
                                                       1e-3, 100.0, 8)
    assert (n_lo, n_hi) == (2, 1)
    s = np.sort(np.linalg.svd(out.U, compute_uv=False))
    np.testing.assert_allclose(s, np.sort([1.0, 1.0, 0.02, 0.7, 1.0, 3.0, 80.0, 1.0]), rtol=1e-9)
    assert s_min == pytest.approx(0.02, rel=1e-9) and s_max == pytest.approx(80.0, rel=1e-9)
    np.testing.assert_allclose(out.V @ out.U, W, rtol=1e-9, atol=1e-9)
    np.testing.assert_allclose(out.U @ out.UinvT.T, np.eye(8), atol=1e-9)


def test_singular_stabilize_cap_and_no_op():
    sig = np.array([1e-5, 2e-5, 3e-5, 0.5, 2.0])
    st, rng = _state_with_singular_values(7, 20, sig)
    _, n_lo, n_hi, s_min, _ = singular_stabilize(st, rng.standard_normal(5), 128, 1e-3, 100.0, 2)
    assert (n_lo, n_hi) == (2, 0) and s_min == pytest.approx(3e-5, rel=1e-8)  # 1e-5, 2e-5 fixed
    st2, rng = _state_with_singular_values(8, 20, np.array([0.5, 1.0, 2.0]))
    out, n_lo, n_hi, _, _ = singular_stabilize(st2, rng.standard_normal(3), 64, 1e-3, 100.0, 4)
    assert (n_lo, n_hi) == (0, 0)
    np.testing.assert_array_equal(out.V, st2.V)
    np.testing.assert_array_equal(out.U, st2.U)


# ---- the sparse input layer of section 2.2 ----

def test_input_layer_brute_force_and_autograd():
    import torch

    from oracle.input_layer import input_forward, input_update
    rng = np.random.default_rng(12)
    D_in, d, m, K = 9, 4, 3, 3
    W1 = rng.standard_normal((D_in, d))
    idx = np.array([[2, 5, 2], [0, -1, 8], [7, 7, 7]], dtype=np.int32)
    val = rng.standard_normal((m, K))
    A = input_forward(W1, idx, val)
    for j in range(m):  # the paper's sum over the K slots, written as loops
        want = np.zeros(d)
        for k in range(K):
            if idx[j, k] >= 0:
                want += val[j, k] * W1[idx[j, k]]
        np.testing.assert_allclose(A[j], want, rtol=0, atol=1e-14)
    G = rng.standard_normal((m, d))
    W1_new = input_update(W1, idx, val, G, 0.3)
    # autograd of sum(A * G) with respect to W1 is the update's direction
    Wt = torch.tensor(W1, dtype=torch.float64, requires_grad=True)
    X = torch.zeros((m, D_in), dtype=torch.float64)
    for j in range(m):
        for k in range(K):
            if idx[j, k] >= 0:
                X[j, idx[j, k]] += val[j, k]
    ((X @ Wt) * torch.tensor(G)).sum().backward()
    np.testing.assert_allclose(W1_new, W1 - 0.3 * Wt.grad.numpy(), rtol=0, atol=1e-13)
    # rows no slot names are unchanged
    for r in (1, 3, 4, 6):
        assert np.array_equal(W1_new[r], W1[r])

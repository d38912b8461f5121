"""Pins of the dense fp64 oracle against things other than itself.

* hand-worked examples (tests/golden/hand_examples.json), exact arithmetic;
* closed forms: W = 0 for every loss; the spherical and Taylor softmax
  normalisation (sum over all D classes of exp(-loss) equals 1);
* the Taylor softmax against the softmax cross-entropy of torch (a library
  routine) for small outputs, where they agree to third order;
* torch.autograd (fp64, CPU) differentiating the loss written from its
  definition: checks grad_H and the W update (dL/dW);
* central finite differences of the oracle's own loss;
* brute force with explicit Python loops on tiny inputs;
* structure of a minibatch: the loss and the update are sums over examples,
  and repeated / empty target slots follow the stated readings.
"""
import json
import os

import numpy as np
import pytest
import torch

from oracle import (dense_step, dense_targets, spherical_softmax_step, squared_error_step,
                    taylor_softmax_step)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")


def _rand_case(seed, D=11, d=4, m=3, K=2, loss="squared"):
    rng = np.random.default_rng(seed)
    W = rng.standard_normal((D, d))
    H = rng.standard_normal((m, d)) / np.sqrt(d)
    idx = np.stack([rng.choice(D, size=K, replace=False) for _ in range(m)]).astype(np.int32)
    val = rng.standard_normal((m, K)) if loss == "squared" else np.ones((m, K))
    return W, H, idx, val


def _golden():
    with open(GOLDEN) as f:
        return json.load(f)


@pytest.mark.parametrize("case", _golden()["examples"], ids=lambda c: c["name"])
def test_hand_examples_squared(case):
    res = squared_error_step(np.array(case["W"], float), np.array(case["H"], float),
                             np.array(case["idx"]), np.array(case["val"], float), case["lr"])
    assert res.loss == pytest.approx(case["L"], abs=1e-12)
    np.testing.assert_allclose(res.grad_H, np.array(case["grad_H"], float), atol=1e-12)
    np.testing.assert_allclose(res.W_new, np.array(case["W_new"], float), atol=1e-12)


def test_hand_example_spherical_softmax():
    case = _golden()["spherical_softmax"][0]
    eps, lr = case["eps"], case["lr"]
    Z = 5.0 + 2 * eps
    L = np.log(Z) - np.log(1 + eps)
    grad_o = np.array([2 / Z - 2 / (1 + eps), 4 / Z])
    W = np.array(case["W"], float)
    res = spherical_softmax_step(W, np.array(case["H"], float), np.array(case["idx"]),
                                 np.array(case["val"], float), lr, eps)
    assert res.loss == pytest.approx(L, abs=1e-14)
    np.testing.assert_allclose(res.grad_H, [[grad_o @ W[:, 0]]], atol=1e-14)
    np.testing.assert_allclose(res.W_new, W - lr * grad_o[:, None] * 1.0, atol=1e-14)


def test_hand_example_taylor_softmax():
    case = _golden()["taylor_softmax"][0]
    res = taylor_softmax_step(np.array(case["W"], float), np.array(case["H"], float),
                              np.array(case["idx"]), np.array(case["val"], float), case["lr"])
    assert res.loss == pytest.approx(np.log(7 / 5), abs=1e-15)
    np.testing.assert_allclose(res.grad_H, [[-8 / 35]], atol=1e-15)
    np.testing.assert_allclose(res.W_new, np.array(case["W_new"], float), atol=1e-15)


def test_squared_zero_W_closed_form():
    _, H, idx, val = _rand_case(1, K=3)
    D, d = 11, 4
    W = np.zeros((D, d))
    res = squared_error_step(W, H, idx, val, 0.05)
    # o = 0: L = sum_j ||y_j||^2, grad_H = 0, W_new = 2 eta Y H (row c gets 2 eta t h_j)
    assert res.loss == pytest.approx(float(np.sum(val ** 2)), rel=1e-14)
    assert np.all(res.grad_H == 0)
    expect = np.zeros((D, d))
    for j in range(H.shape[0]):
        for k in range(idx.shape[1]):
            expect[idx[j, k]] += 2 * 0.05 * val[j, k] * H[j]
    np.testing.assert_allclose(res.W_new, expect, atol=1e-15)


def test_spherical_softmax_zero_W_closed_form():
    _, H, idx, val = _rand_case(2, D=13, K=1, loss="spherical_softmax")
    W = np.zeros((13, 4))
    res = spherical_softmax_step(W, H, idx, val, 0.1, 1e-3)
    # every output is 0, so every class has probability eps / (D eps) = 1/D
    np.testing.assert_allclose(res.per_example, np.log(13.0), rtol=1e-14)
    assert np.all(res.grad_H == 0) and np.all(res.W_new == 0)


def test_spherical_softmax_normalises_over_all_classes():
    W, H, _, _ = _rand_case(3, D=9, d=3, m=2, K=1, loss="spherical_softmax")
    for eps in (1e-3, 0.5):
        for j in range(2):
            tot = 0.0
            for c in range(9):
                res = spherical_softmax_step(W, H[j:j + 1], np.array([[c]]), np.ones((1, 1)),
                                             0.1, eps)
                tot += np.exp(-res.loss)
            assert tot == pytest.approx(1.0, abs=1e-13)


def test_taylor_softmax_zero_W_closed_form():
    _, H, idx, val = _rand_case(4, D=13, K=2, loss="taylor_softmax")
    W = np.zeros((13, 4))
    res = taylor_softmax_step(W, H, idx, val, 0.1)
    # o = 0, f(0) = 1: every class has probability 1/D; grad_O = (T/D) 1_D - Y (dl/da = -t
    # since f'(0)/f(0) = 1), so grad_H = W^T grad_O = 0 and W_new = -eta grad_O H
    np.testing.assert_allclose(res.per_example, val.sum(axis=1) * np.log(13.0), rtol=1e-14)
    assert np.all(res.grad_H == 0)
    gO = val.sum(axis=1)[None, :] / 13.0 - dense_targets(13, idx, val)
    np.testing.assert_allclose(res.W_new, -0.1 * gO @ H, atol=1e-16)


def test_taylor_softmax_normalises_over_all_classes():
    W, H, _, _ = _rand_case(8, D=9, d=3, m=2, K=1, loss="taylor_softmax")
    W *= 3.0  # large outputs, negative ones included: f stays positive
    for j in range(2):
        tot = sum(np.exp(-taylor_softmax_step(W, H[j:j + 1], np.array([[c]]), np.ones((1, 1)),
                                               0.1).loss) for c in range(9))
        assert tot == pytest.approx(1.0, abs=1e-13)


@pytest.mark.parametrize("scale", [1e-2, 3e-2])
def test_taylor_softmax_agrees_with_softmax_to_third_order(scale):
    # log f(x) = x - x^3/6 + O(x^4) and log sum f = logsumexp + O(max |o|^3): the two losses
    # differ by at most about max|o|^3 / 3 per unit of target weight
    W, H, idx, val = _rand_case(9, D=40, d=6, m=3, K=2, loss="taylor_softmax")
    W *= scale / np.abs(W @ H.T).max()
    res = taylor_softmax_step(W, H, idx, val, 0.1)
    logp = torch.log_softmax(torch.tensor(W @ H.T), dim=0).numpy()
    for j in range(3):
        ce = -sum(val[j, k] * logp[idx[j, k], j] for k in range(2))
        assert abs(res.per_example[j] - ce) <= 2 * 0.5 * scale ** 3
        assert abs(res.per_example[j] - ce) < 1e-2 * abs(ce)


def _torch_loss(Wt, Ht, idx, val, loss, eps):
    D = Wt.shape[0]
    O = Wt @ Ht.T
    if loss == "squared":
        Y = torch.tensor(dense_targets(D, idx, val))
        return ((O - Y) ** 2).sum()
    tot = 0
    if loss == "taylor_softmax":  # f over every output, the normaliser summed explicitly
        F = 1 + O + O * O / 2
        denom = F.sum(dim=0)
        for j in range(idx.shape[0]):
            for k in range(idx.shape[1]):
                c = int(idx[j, k])
                if c >= 0:
                    tot = tot - val[j, k] * torch.log(F[c, j] / denom[j])
        return tot
    denom = (O * O + eps).sum(dim=0)
    for j in range(idx.shape[0]):
        for k in range(idx.shape[1]):
            c = int(idx[j, k])
            if c >= 0:
                tot = tot - val[j, k] * torch.log((O[c, j] ** 2 + eps) / denom[j])
    return tot


@pytest.mark.parametrize("loss", ["squared", "spherical_softmax", "taylor_softmax"])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_autograd(loss, seed):
    W, H, idx, val = _rand_case(seed, D=17, d=5, m=4, K=3, loss=loss)
    lr, eps = 0.03, 1e-3
    res = dense_step(W, H, idx, val, lr, loss, eps)
    Wt = torch.tensor(W, requires_grad=True)
    Ht = torch.tensor(H, requires_grad=True)
    Lt = _torch_loss(Wt, Ht, idx, val, loss, eps)
    Lt.backward()
    assert res.loss == pytest.approx(Lt.item(), rel=1e-13)
    np.testing.assert_allclose(res.grad_H, Ht.grad.numpy(), rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(res.W_new, W - lr * Wt.grad.numpy(), rtol=1e-11, atol=1e-12)


@pytest.mark.parametrize("loss", ["squared", "spherical_softmax", "taylor_softmax"])
def test_finite_differences(loss):
    W, H, idx, val = _rand_case(7, D=8, d=3, m=2, K=2, loss=loss)
    lr, eps, h = 0.05, 1e-2, 1e-6
    res = dense_step(W, H, idx, val, lr, loss, eps)

    def L(W_, H_):
        return dense_step(W_, H_, idx, val, lr, loss, eps).loss

    for (j, c) in [(0, 0), (1, 2), (0, 1)]:
        Hp, Hm = H.copy(), H.copy()
        Hp[j, c] += h
        Hm[j, c] -= h
        fd = (L(W, Hp) - L(W, Hm)) / (2 * h)
        assert res.grad_H[j, c] == pytest.approx(fd, rel=1e-6, abs=1e-7)
    dW = (W - res.W_new) / lr
    for (r, c) in [(idx[0, 0], 0), (idx[1, 1], 2), (5, 1)]:
        Wp, Wm = W.copy(), W.copy()
        Wp[r, c] += h
        Wm[r, c] -= h
        fd = (L(Wp, H) - L(Wm, H)) / (2 * h)
        assert dW[r, c] == pytest.approx(fd, rel=1e-6, abs=1e-7)


def test_brute_force_loops_squared():
    W, H, idx, val = _rand_case(11, D=7, d=3, m=2, K=2)
    D, d = W.shape
    m, K = idx.shape
    L = 0.0
    for j in range(m):
        for i in range(D):
            o = 0.0
            for c in range(d):
                o += W[i, c] * H[j, c]
            y = 0.0
            for k in range(K):
                if idx[j, k] == i:
                    y += val[j, k]
            L += (o - y) ** 2
    assert squared_error_step(W, H, idx, val, 0.1).loss == pytest.approx(L, rel=1e-13)


@pytest.mark.parametrize("loss", ["squared", "spherical_softmax", "taylor_softmax"])
def test_minibatch_is_sum_of_examples(loss):
    W, H, idx, val = _rand_case(5, D=10, d=4, m=3, K=2, loss=loss)
    lr = 0.02
    full = dense_step(W, H, idx, val, lr, loss)
    dW = np.zeros_like(W)
    Ls = 0.0
    for j in range(3):
        one = dense_step(W, H[j:j + 1], idx[j:j + 1], val[j:j + 1], lr, loss)
        Ls += one.loss
        dW += one.W_new - W
        np.testing.assert_allclose(full.grad_H[j], one.grad_H[0], rtol=1e-12, atol=1e-14)
    assert full.loss == pytest.approx(Ls, rel=1e-13)
    np.testing.assert_allclose(full.W_new, W + dW, rtol=1e-12, atol=1e-14)


def test_example_and_slot_order_invariance():
    W, H, idx, val = _rand_case(6, D=12, d=4, m=4, K=3)
    base = squared_error_step(W, H, idx, val, 0.01)
    perm = np.array([2, 0, 3, 1])
    p = squared_error_step(W, H[perm], idx[perm], val[perm], 0.01)
    assert p.loss == pytest.approx(base.loss, rel=1e-13)
    np.testing.assert_allclose(p.grad_H, base.grad_H[perm], rtol=1e-12)
    np.testing.assert_allclose(p.W_new, base.W_new, rtol=1e-12, atol=1e-15)
    sp = squared_error_step(W, H, idx[:, ::-1].copy(), val[:, ::-1].copy(), 0.01)
    np.testing.assert_allclose(sp.W_new, base.W_new, rtol=1e-12, atol=1e-15)


@pytest.mark.parametrize("loss", ["spherical_softmax", "taylor_softmax"])
def test_repeated_index_adds_values_spherical(loss):
    # a spherical-family loss with two slots of the same class c and weights t1, t2 equals one
    # slot with weight t1 + t2 (the per-slot sum reading); an empty slot adds nothing
    W, H, _, _ = _rand_case(8, D=6, d=3, m=1, K=1, loss=loss)
    a = dense_step(W, H, np.array([[4, 4, -1]]), np.array([[0.25, 0.5, 9.0]]), 0.1, loss, 1e-3)
    b = dense_step(W, H, np.array([[4]]), np.array([[0.75]]), 0.1, loss, 1e-3)
    assert a.loss == pytest.approx(b.loss, rel=1e-14)
    np.testing.assert_allclose(a.grad_H, b.grad_H, rtol=1e-13)
    np.testing.assert_allclose(a.W_new, b.W_new, rtol=1e-13)


def test_index_out_of_range_rejected():
    W, H, idx, val = _rand_case(9)
    idx[0, 0] = W.shape[0]
    with pytest.raises(ValueError):
        squared_error_step(W, H, idx, val, 0.1)

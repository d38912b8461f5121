"""Dense fp64 oracle: the plain definition of one minibatch step (test infrastructure only).

W is held explicitly (D x d).  For a minibatch H (m x d here, one example per
row; the paper's d x m H with one example per column) and K-sparse targets
(idx, val) it computes the full output O = W H^T (D x m), the loss, the
gradient of the loss with respect to H and the gradient-descent update of W.
Nothing here uses Q, U, U^{-T} or any other piece of the factored method.

Sources in the paper:
  squared error    -- section 2.1 (L = ||o - y||^2), section 2.3 (the three
                      O(Dd) operations), section 3.2 (dL/dW = 2 (Wh - y) h^T and
                      W <- W - 2 eta (Wh - y) h^T); minibatch loss is the sum
                      over the m examples (Algorithm 3, outputs).
  spherical family -- section 4: the naive forward steps (o = W h, q = ||o||^2,
                      s = sum(o), l = loss(q, s, K, o_K, y_K)) and the naive
                      backward steps (grad_o = 2 o dl/dq + 1_D dl/ds + y_ring,
                      grad_h = W^T grad_o, W <- W - eta grad_o h^T), in the
                      minibatch form of eq. gen-grad-O and eq. gen-update-W.
  spherical softmax -- the paper names it but never defines it.  The reading
                      used everywhere here: for example j with target slots
                      (c_k, t_k), l_j = -sum_k t_k log((o_{c_k}^2 + eps) /
                      sum_i (o_i^2 + eps)); the denominator is q_j + D eps and
                      the loss does not depend on s.
  Taylor softmax   -- also named in section 4 and never defined.  The reading:
                      the softmax with exp replaced by its second-order Taylor
                      polynomial f(x) = 1 + x + x^2/2 (positive everywhere, so
                      every output is a probability),
                      l_j = -sum_k t_k log(f(o_{c_k}) / sum_i f(o_i)); the
                      denominator is sum_i f(o_i) = D + s_j + q_j / 2, so the
                      loss depends on both q and s (dl/dq = T / (2 Z),
                      dl/ds = T / Z with T = sum_k t_k, Z = D + s + q/2).
Target representation: (index, value) pairs (section 2.1, section 4.1.4), with
-1 marking an empty slot; an index repeated inside one example adds its values
(y = sum_k t_k onehot(c_k)).
"""
from __future__ import annotations

from typing import NamedTuple

import numpy as np

F64 = np.float64


class StepResult(NamedTuple):
    loss: float              # sum over the minibatch of the per-example losses
    grad_H: np.ndarray       # m x d, d loss / d H
    W_new: np.ndarray        # D x d, W - lr * d loss / d W
    per_example: np.ndarray  # m, per-example losses


def _check_idx(D: int, idx: np.ndarray) -> None:
    if idx.size and (idx.min() < -1 or idx.max() >= D):
        raise ValueError("target index outside [-1, D)")


def dense_targets(D: int, idx: np.ndarray, val: np.ndarray) -> np.ndarray:
    """Y (D x m): column j holds sum_k val[j,k] onehot(idx[j,k]); -1 slots are skipped."""
    idx = np.asarray(idx)
    val = np.asarray(val, dtype=F64)
    _check_idx(D, idx)
    m, K = idx.shape
    Y = np.zeros((D, m), dtype=F64)
    rows = idx.reshape(-1).astype(np.int64)
    cols = np.repeat(np.arange(m), K)
    keep = rows >= 0
    np.add.at(Y, (rows[keep], cols[keep]), val.reshape(-1)[keep])
    return Y


def squared_error_step(W, H, idx, val, lr) -> StepResult:
    """L = ||W H^T - Y||_F^2, grad_H = 2 (O - Y)^T W, W_new = W - 2 lr (O - Y) H."""
    W = np.asarray(W, dtype=F64)
    H = np.asarray(H, dtype=F64)
    lr = F64(lr)
    D = W.shape[0]
    Y = dense_targets(D, idx, val)
    O = W @ H.T                       # D x m, the O(Dd)-per-example output
    R = O - Y
    per = np.sum(R * R, axis=0)
    grad_H = 2.0 * (R.T @ W)          # m x d
    W_new = W - 2.0 * lr * (R @ H)
    return StepResult(float(per.sum()), grad_H, W_new, per)


def spherical_softmax_step(W, H, idx, val, lr, eps) -> StepResult:
    """Spherical softmax through the naive steps of section 4 (dl/ds = 0)."""
    W = np.asarray(W, dtype=F64)
    H = np.asarray(H, dtype=F64)
    idx = np.asarray(idx)
    val = np.asarray(val, dtype=F64)
    lr = F64(lr)
    eps = F64(eps)
    D = W.shape[0]
    _check_idx(D, idx)
    m, K = idx.shape
    O = W @ H.T                       # D x m
    q = np.sum(O * O, axis=0)         # q_j = ||o_j||^2
    denom = q + D * eps               # sum_i (o_ij^2 + eps)
    per = np.zeros(m, dtype=F64)
    dl_dq = np.zeros(m, dtype=F64)
    y_ring = np.zeros((D, m), dtype=F64)   # sparse dl/da placed at the target rows
    for j in range(m):
        for k in range(K):
            c = int(idx[j, k])
            if c < 0:
                continue
            t = val[j, k]
            a = O[c, j]
            per[j] -= t * (np.log(a * a + eps) - np.log(denom[j]))
            dl_dq[j] += t / denom[j]
            y_ring[c, j] += -2.0 * t * a / (a * a + eps)
    grad_O = 2.0 * O * dl_dq[None, :] + y_ring
    grad_H = grad_O.T @ W
    W_new = W - lr * (grad_O @ H)
    return StepResult(float(per.sum()), grad_H, W_new, per)


def taylor_softmax_step(W, H, idx, val, lr) -> StepResult:
    """Taylor softmax through the naive steps of section 4, with dl/ds nonzero:
    grad_O = 2 O diag(dl/dq) + 1_D (dl/ds)^T + Yring (eq. gen-grad-O)."""
    W = np.asarray(W, dtype=F64)
    H = np.asarray(H, dtype=F64)
    idx = np.asarray(idx)
    val = np.asarray(val, dtype=F64)
    lr = F64(lr)
    D = W.shape[0]
    _check_idx(D, idx)
    m, K = idx.shape
    O = W @ H.T                       # D x m
    q = np.sum(O * O, axis=0)         # q_j = ||o_j||^2
    s = np.sum(O, axis=0)             # s_j = sum(o_j)
    Z = D + s + 0.5 * q               # sum_i f(o_ij)
    per = np.zeros(m, dtype=F64)
    dl_dq = np.zeros(m, dtype=F64)
    dl_ds = np.zeros(m, dtype=F64)
    y_ring = np.zeros((D, m), dtype=F64)
    for j in range(m):
        for k in range(K):
            c = int(idx[j, k])
            if c < 0:
                continue
            t = val[j, k]
            a = O[c, j]
            fa = 1.0 + a + 0.5 * a * a
            per[j] -= t * (np.log(fa) - np.log(Z[j]))
            dl_dq[j] += t / (2.0 * Z[j])
            dl_ds[j] += t / Z[j]
            y_ring[c, j] -= t * (1.0 + a) / fa
    grad_O = 2.0 * O * dl_dq[None, :] + dl_ds[None, :] + y_ring
    grad_H = grad_O.T @ W
    W_new = W - lr * (grad_O @ H)
    return StepResult(float(per.sum()), grad_H, W_new, per)


def dense_step(W, H, idx, val, lr, loss: str = "squared", eps: float = 1e-3) -> StepResult:
    if loss == "squared":
        return squared_error_step(W, H, idx, val, lr)
    if loss == "spherical_softmax":
        return spherical_softmax_step(W, H, idx, val, lr, eps)
    if loss == "taylor_softmax":
        return taylor_softmax_step(W, H, idx, val, lr)
    raise ValueError(loss)

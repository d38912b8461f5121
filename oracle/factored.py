"""fp64 factored mirror of the paper's algorithms (test infrastructure only).

W is never formed: it is represented as V U (+ 1_D omega^T for losses that use
s = sum(o), eq. gen-Wfact) with the bookkeeping matrices Q = W^T W, U^{-T} and
w_bar = W^T 1_D.  Two step functions follow the paper's tables in their order
and notation, with the paper's H = d x m (here Hp = H^T, H being the m x d
row-major minibatch):

  alg3_step -- Algorithm 3 (minibatch, squared error), steps 1..8.
  alg4_step -- Algorithm 4 (minibatch, general spherical loss).  For squared
               error and the spherical softmax dl/ds = 0 and omega stays 0 (the
               closing remark of section 4.8); for the Taylor softmax every row
               of the table runs: s = H^T w_bar, h~ = H^T omega, the omega and
               w_bar updates and the grad_s terms of Z^ and M.

The U^{-T} update of Algorithm 4 is only named in the paper (section 4.7: use
the Woodbury identity).  The form used here: with S = diag(grad_q)^{1/2},
U_new = U (I - 2 eta H S S H^T), so by Woodbury
    U_new^{-T} = U^{-T} + 2 eta (U^{-T} H) S C^{-1} S H^T,  C = I_m - 2 eta S H^T H S,
which is Algorithm 3 step 6 when S = I and eq. updateU-T (Sherman-Morrison)
when m = 1.

The mirror shares nothing with the HIP path.  It is pinned against the dense
oracle (section 3.2, 3.4 and 4.4 proofs of exactness) by the test suite.
"""
from __future__ import annotations

import dataclasses

import numpy as np

F64 = np.float64


@dataclasses.dataclass
class FactoredState:
    V: np.ndarray      # D x d
    U: np.ndarray      # d x d
    UinvT: np.ndarray  # d x d, (U^{-1})^T
    Q: np.ndarray      # d x d, W^T W
    omega: np.ndarray = None  # d, W = V U + 1_D omega^T (eq. gen-Wfact)
    wbar: np.ndarray = None   # d, W^T 1_D

    def __post_init__(self):
        d = self.U.shape[0]
        if self.omega is None:
            self.omega = np.zeros(d, dtype=F64)
        if self.wbar is None:
            self.wbar = (self.V @ self.U + self.omega[None, :]).sum(axis=0)

    def W(self) -> np.ndarray:
        return self.V @ self.U + self.omega[None, :]

    def copy(self) -> "FactoredState":
        return FactoredState(self.V.copy(), self.U.copy(), self.UinvT.copy(), self.Q.copy(),
                             self.omega.copy(), self.wbar.copy())


def factored_init(V0, U0=None) -> FactoredState:
    """Algorithm 1 and the initialisation of section 4.8: V = V0, U = I (or a given U),
    U^{-T} = inv(U)^T, Q = W^T W (= V^T V for U = I), omega = 0, w_bar = W^T 1_D
    (= rowsum(V) for U = I)."""
    V = np.array(V0, dtype=F64, copy=True)
    d = V.shape[1]
    if U0 is None:
        U = np.eye(d, dtype=F64)
        UinvT = np.eye(d, dtype=F64)
        Q = V.T @ V
        wbar = V.sum(axis=0)
    else:
        U = np.array(U0, dtype=F64, copy=True)
        UinvT = np.linalg.inv(U).T
        W = V @ U
        Q = W.T @ W
        wbar = W.sum(axis=0)
    return FactoredState(V, U, UinvT, Q, np.zeros(d, dtype=F64), wbar)


def _slots(idx):
    m, K = idx.shape
    for j in range(m):
        for k in range(K):
            c = int(idx[j, k])
            if c >= 0:
                yield j, k, c


def _sparse_gram(idx, w) -> np.ndarray:
    """m x m matrix with entries sum_{k,k'} w[i,k] w[j,k'] [idx[i,k] == idx[j,k']] (dot products of
    two K-sparse columns, the Y^T Y / Yring^T Yring terms; -1 slots never match)."""
    m, K = idx.shape
    G = np.zeros((m, m), dtype=F64)
    for i in range(m):
        for j in range(m):
            s = 0.0
            for k in range(K):
                if idx[i, k] < 0:
                    continue
                for kk in range(K):
                    if idx[i, k] == idx[j, kk]:
                        s += w[i, k] * w[j, kk]
            G[i, j] = s
    return G


def alg3_step(st: FactoredState, H, idx, val, lr):
    """Algorithm 3 (squared error).  Updates st in place; returns (L, grad_H m x d, intermediates)."""
    Hp = np.asarray(H, dtype=F64).T            # d x m
    idx = np.asarray(idx)
    T = np.asarray(val, dtype=F64)
    lr = F64(lr)
    m = Hp.shape[1]
    V, U, UinvT, Q = st.V, st.U, st.UinvT, st.Q
    # 1: H^ = Q H
    Hhat = Q @ Hp
    # 2: Y^ = U^T (V^T Y), V^T Y gathered from the K target rows of V
    VtY = np.zeros_like(Hp)
    for j, k, c in _slots(idx):
        VtY[:, j] += T[j, k] * V[c]
    Yhat = U.T @ VtY
    # 3: grad_H = 2 (H^ - Y^)
    grad = 2.0 * (Hhat - Yhat)
    # 4a: M = H^T H^ - (Y^T H + H^T Y^) + Y^T Y ; 4b: L = Tr M
    YtY = _sparse_gram(idx, T)
    M = Hp.T @ Hhat - (Yhat.T @ Hp + Hp.T @ Yhat) + YtY
    L = float(np.trace(M))
    # 5: U <- U - 2 eta (U H) H^T
    U_new = U - 2.0 * lr * (U @ Hp) @ Hp.T
    # 6: U^{-T} <- U^{-T} - (U^{-T} H) ((H^T H - I/(2 eta))^{-1} H^T)   [Woodbury]
    X = UinvT @ Hp
    Cw = Hp.T @ Hp - np.eye(m) / (2.0 * lr)
    UinvT_new = UinvT - X @ np.linalg.solve(Cw, Hp.T)
    # 7: V <- V + 2 eta Y (U_new^{-T} H)^T, with the fresh U^{-T}
    P = UinvT_new @ Hp
    for j, k, c in _slots(idx):
        V[c] += 2.0 * lr * T[j, k] * P[:, j]
    # 8: Q <- Q - eta (H grad^T + grad H^T) + 4 eta^2 (H M) H^T
    Q_new = Q - lr * (Hp @ grad.T + grad @ Hp.T) + 4.0 * lr * lr * (Hp @ M) @ Hp.T
    st.U, st.UinvT, st.Q = U_new, UinvT_new, Q_new
    inter = dict(Hhat=Hhat, Yhat=Yhat, M=M, X=X, P=P, VtY=VtY)
    return L, grad.T.copy(), inter


def spherical_loss(loss: str, q, s, a, t, valid, D: int, eps: float, idx_row):
    """One example's loss l(q, s, K, a, t) and its partial derivatives (dl/dq, dl/ds, dl/da).

    squared:            l = q - 2 a.t + ||y||^2           (section 4, squared error as a member)
    spherical softmax:  l = sum_k t_k [log(q + D eps) - log(a_k^2 + eps)]
    Taylor softmax:     l = sum_k t_k [log(D + s + q/2) - log(1 + a_k + a_k^2/2)]
    """
    K = len(a)
    dA = np.zeros(K, dtype=F64)
    if loss == "squared":
        yy = 0.0
        for k in range(K):
            if not valid[k]:
                continue
            for kk in range(K):
                if valid[kk] and idx_row[k] == idx_row[kk]:
                    yy += t[k] * t[kk]
        at = sum(a[k] * t[k] for k in range(K) if valid[k])
        for k in range(K):
            if valid[k]:
                dA[k] = -2.0 * t[k]
        return q - 2.0 * at + yy, 1.0, 0.0, dA
    if loss == "spherical_softmax":
        z = q + D * eps
        l = 0.0
        dq = 0.0
        for k in range(K):
            if not valid[k]:
                continue
            l += t[k] * (np.log(z) - np.log(a[k] * a[k] + eps))
            dq += t[k] / z
            dA[k] = -2.0 * t[k] * a[k] / (a[k] * a[k] + eps)
        return l, dq, 0.0, dA
    if loss == "taylor_softmax":
        z = D + s + 0.5 * q
        l = 0.0
        dq = 0.0
        ds = 0.0
        for k in range(K):
            if not valid[k]:
                continue
            f = 1.0 + a[k] + 0.5 * a[k] * a[k]
            l += t[k] * (np.log(z) - np.log(f))
            dq += t[k] / (2.0 * z)
            ds += t[k] / z
            dA[k] = -t[k] * (1.0 + a[k]) / f
        return l, dq, ds, dA
    raise ValueError(loss)


def alg4_step(st: FactoredState, H, idx, val, lr, loss: str = "squared", eps: float = 1e-3):
    """Algorithm 4, its rows in order.  Updates st in place; returns (L, grad_H, intermediates)."""
    Hp = np.asarray(H, dtype=F64).T            # d x m
    idx = np.asarray(idx)
    T = np.asarray(val, dtype=F64)
    lr = F64(lr)
    d, m = Hp.shape
    K = idx.shape[1]
    V, U, UinvT, Q, omega, wbar = st.V, st.U, st.UinvT, st.Q, st.omega, st.wbar
    D = V.shape[0]
    Hhat = Q @ Hp                              # H^ = Q H
    Mhat = Hp.T @ Hhat                         # M^ = H^T H^
    q = np.diag(Mhat).copy()                   # q = diag(M^)
    s = Hp.T @ wbar                            # s = H^T w_bar (eq. svec)
    Htil = U @ Hp                              # H~ = U H
    hw = Hp.T @ omega                          # h~ = H^T omega (eq. gen-htilde)
    A = np.zeros((K, m), dtype=F64)            # A_kj = H~_j . V_{K_kj} + h~_j
    for j, k, c in _slots(idx):
        A[k, j] = Htil[:, j] @ V[c] + hw[j]
    per = np.zeros(m, dtype=F64)
    dq = np.zeros(m, dtype=F64)
    ds = np.zeros(m, dtype=F64)
    dA = np.zeros((K, m), dtype=F64)
    for j in range(m):
        valid = idx[j] >= 0
        per[j], dq[j], ds[j], dA[:, j] = spherical_loss(loss, q[j], s[j], A[:, j], T[j], valid, D,
                                                        eps, idx[j])
    L = float(per.sum())
    ybar = np.array([sum(dA[k, j] for k in range(K) if idx[j, k] >= 0) for j in range(m)],
                    dtype=F64)                 # y_bar = rowsum(grad_A) (eq. ybar)
    VtYr = np.zeros_like(Hp)                   # V^T Yring, K rows of V per example
    for j, k, c in _slots(idx):
        VtYr[:, j] += dA[k, j] * V[c]
    # Z^ = w_bar grad_s^T + U^T (V^T Yring) + omega y_bar^T (eq. gen-Zhat-fact)
    Zhat = np.outer(wbar, ds) + U.T @ VtYr + np.outer(omega, ybar)
    grad = 2.0 * Hhat * dq[None, :] + Zhat     # grad_H = 2 H^ diag(grad_q) + Z^
    # U <- U - 2 eta (U H) diag(grad_q) H^T
    U_new = U - 2.0 * lr * (Htil * dq[None, :]) @ Hp.T
    # U^{-T} by Woodbury (see module docstring)
    sq = np.sqrt(dq)
    X = UinvT @ Hp
    N = Hp.T @ Hp
    C = np.eye(m) - 2.0 * lr * (sq[:, None] * N * sq[None, :])
    B = sq[:, None] * np.linalg.solve(C, np.diag(sq))
    UinvT_new = UinvT + 2.0 * lr * (X @ B) @ Hp.T
    # omega <- omega - eta H (2 diag(grad_q) h~ + grad_s) (eq. gen-update-omega)
    omega_new = omega - lr * Hp @ (2.0 * dq * hw + ds)
    # V <- V - eta Yring (U_new^{-T} H)^T
    P = UinvT_new @ Hp
    for j, k, c in _slots(idx):
        V[c] -= lr * dA[k, j] * P[:, j]
    # w_bar <- w_bar - eta H (2 diag(grad_q) H^T w_bar + D grad_s + y_bar) (eq. gen-update-wbar,
    # in the form of its derivation and of Algorithm 4's table)
    wbar_new = wbar - lr * Hp @ (2.0 * dq * s + D * ds + ybar)
    # M (eq. gen-M) and Q <- Q - eta grad H^T - eta H grad^T + eta^2 (H M) H^T
    YrYr = _sparse_gram(idx, dA.T)
    HZ = dq[:, None] * (Hp.T @ Zhat)
    M = (4.0 * dq[:, None] * Mhat * dq[None, :] + D * np.outer(ds, ds) + YrYr
         + np.outer(ds, ybar) + np.outer(ybar, ds) + 2.0 * HZ + 2.0 * HZ.T)
    Q_new = Q - lr * grad @ Hp.T - lr * Hp @ grad.T + lr * lr * (Hp @ M) @ Hp.T
    st.U, st.UinvT, st.Q, st.omega, st.wbar = U_new, UinvT_new, Q_new, omega_new, wbar_new
    inter = dict(Hhat=Hhat, Htil=Htil, q=q, s=s, hw=hw, A=A, dq=dq, ds=ds, dA=dA, ybar=ybar,
                 G=VtYr, Zhat=Zhat, M=M, N=N, C=C, B=B, X=X, P=P, per_example=per)
    return L, grad.T.copy(), inter


def factored_step(st: FactoredState, H, idx, val, lr, loss: str = "squared", eps: float = 1e-3):
    """One factored step (Algorithm 4 form for both losses)."""
    return alg4_step(st, H, idx, val, lr, loss, eps)

"""fp64 oracle of the numerical stabilisation of section 5 -- TEST INFRASTRUCTURE ONLY.

W = V U is never changed by any of these operations; they act on how it is
split between V and U, and on the bookkeeping inverse U^{-T}:

  restore_pristine   -- section 5.1: V <- V U, U <- I, U^{-T} <- I (Q = W^T W kept).
  reinvert           -- section 5.3, last paragraph: U^{-T} recomputed from U alone
                        by Gaussian elimination (LAPACK's LU with partial pivoting).
  power_iteration    -- section 5.3: the left singular vector of a d x d matrix A
                        for its largest singular value, by repeated u <- A A^T u with
                        normalisation, and that singular value ||A^T u||.
  smallest_singular  -- section 5.3: the same on U^{-T}, whose largest singular value
                        is 1 / sigma_min(U) with U's left singular vector.
  largest_singular   -- the same on U.
  fix_singular_value -- Algorithm 5's procedure: with alpha = (s* - s) / s and
                        beta = -alpha / (1 + alpha), U <- U + alpha u (U^T u)^T,
                        V <- V + beta (V u) u^T, U^{-T} <- U^{-T} + beta u (U^{-1} u)^T
                        (U^{-1} = (U^{-T})^T before the update).
  singular_stabilize -- section 5.3's loop: U^{-T} recomputed, then the smallest
                        singular value found and set to 1 while it is below the safe
                        range, then the largest while it is above.

Start vectors of the power iteration are inputs (seeded by the caller).  Shares
nothing with the HIP path.
"""
from __future__ import annotations

import numpy as np

from .factored import FactoredState

F64 = np.float64


def restore_pristine(st: FactoredState) -> FactoredState:
    """Section 5.1: move U into V; U and U^{-T} become the identity, Q is unchanged."""
    d = st.U.shape[0]
    return FactoredState(st.V @ st.U, np.eye(d, dtype=F64), np.eye(d, dtype=F64), st.Q.copy(),
                         st.omega.copy(), st.wbar.copy())


def reinvert(st: FactoredState) -> FactoredState:
    """Section 5.3: U^{-T} from U by Gaussian elimination (no use of the carried value)."""
    return FactoredState(st.V.copy(), st.U.copy(), np.linalg.inv(st.U).T, st.Q.copy(),
                         st.omega.copy(), st.wbar.copy())


def power_iteration(A, u0, iters: int):
    """Section 5.3: iters rounds of u <- A (A^T u) / ||A (A^T u)|| from u0.

    Returns (u, ||A^T u||): the left singular vector of A for its largest singular
    value and that value, once the iteration has converged."""
    A = np.asarray(A, dtype=F64)
    u = np.asarray(u0, dtype=F64) / np.linalg.norm(u0)
    for _ in range(iters):
        v = A @ (A.T @ u)
        u = v / np.linalg.norm(v)
    return u, float(np.linalg.norm(A.T @ u))


def smallest_singular(st: FactoredState, u0, iters: int):
    """sigma_min(U) and its left singular vector, from the largest singular value of
    U^{-T} = Ubar diag(1/sigma) Vbar^T (same left singular vectors as U)."""
    u, s_inv = power_iteration(st.UinvT, u0, iters)
    return u, 1.0 / s_inv


def largest_singular(st: FactoredState, u0, iters: int):
    """sigma_max(U) and its left singular vector."""
    return power_iteration(st.U, u0, iters)


def fix_singular_value(st: FactoredState, sigma: float, u, target: float = 1.0) -> FactoredState:
    """Algorithm 5, fix-singular-value: the singular value sigma of U along its left
    singular vector u becomes target; V takes the inverse rank-one factor so that
    V U is unchanged, and U^{-T} its rank-one update."""
    u = np.asarray(u, dtype=F64)
    alpha = (target - sigma) / sigma
    beta = -alpha / (1.0 + alpha)
    U = st.U + alpha * np.outer(u, st.U.T @ u)
    V = st.V + beta * np.outer(st.V @ u, u)
    UinvT = st.UinvT + beta * np.outer(u, st.UinvT.T @ u)
    return FactoredState(V, U, UinvT, st.Q.copy(), st.omega.copy(), st.wbar.copy())


def singular_stabilize(st: FactoredState, u0, iters: int, lo: float, hi: float, max_fixes: int):
    """Section 5.3's procedure: recompute U^{-T}; while sigma_min(U) < lo (and fewer than
    max_fixes corrections in this direction), set it to 1; then the same for
    sigma_max(U) > hi.  Returns (state, fixes_min, fixes_max, sigma_min, sigma_max) with
    the last values the searches found."""
    st = reinvert(st)
    n_lo = 0
    while True:
        u, s = smallest_singular(st, u0, iters)
        if s >= lo or n_lo >= max_fixes:
            s_min = s
            break
        st = fix_singular_value(st, s, u, 1.0)
        n_lo += 1
    n_hi = 0
    while True:
        u, s = largest_singular(st, u0, iters)
        if s <= hi or n_hi >= max_fixes:
            s_max = s
            break
        st = fix_singular_value(st, s, u, 1.0)
        n_hi += 1
    return st, n_lo, n_hi, s_min, s_max

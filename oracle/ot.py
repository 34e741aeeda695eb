"""Exact transport linear programs, solved with scipy's HiGHS (Sec. 3.1 Eq. 2,
Sec. 3.2 Eq. 5, Sec. 3.5 Eq. 11, Sec. 4.2 Eq. 19-20).  Test infrastructure
only: these pin the readings used by ``sgs`` and ``lite`` on tiny inputs.

Every program minimises <C, P> over P >= 0 (m x n) with C given source-major.
"""
from __future__ import annotations

import numpy as np
from scipy.optimize import linprog


def _solve(C, A_eq=None, b_eq=None, A_ub=None, b_ub=None, zero_mask=None):
    C = np.asarray(C, np.float64)
    m, n = C.shape
    bounds = [(0.0, 0.0) if (zero_mask is not None and zero_mask[i, j]) else (0.0, None)
              for i in range(m) for j in range(n)]
    res = linprog(C.ravel(), A_ub=A_ub, b_ub=b_ub, A_eq=A_eq, b_eq=b_eq,
                  bounds=bounds, method="highs")
    if res.status != 0:
        raise RuntimeError(res.message)
    return float(res.fun), res.x.reshape(m, n)


def _row_sums(m, n):
    A = np.zeros((m, m * n))
    for i in range(m):
        A[i, i * n:(i + 1) * n] = 1.0
    return A


def _col_sums(m, n):
    A = np.zeros((n, m * n))
    for j in range(n):
        A[j, j::n] = 1.0
    return A


def ot_lp(C, u, v):
    """Balanced OT (Eq. 2): P 1 = u, P^T 1 = v."""
    m, n = np.shape(C)
    A = np.vstack([_row_sums(m, n), _col_sums(m, n)])
    return _solve(C, A_eq=A, b_eq=np.concatenate([u, v]))


def sot_lp(C, u, v):
    """Semi-relaxed OT (Eq. 11): P 1 = u, P^T 1 <= v."""
    m, n = np.shape(C)
    return _solve(C, A_eq=_row_sums(m, n), b_eq=np.asarray(u, np.float64),
                  A_ub=_col_sums(m, n), b_ub=np.asarray(v, np.float64))


def free_source_lp(C, v):
    """Transport with the source masses left free: P^T 1 = v only.  This is
    the epsilon -> 0, free-source limit that the greedy's set function uses."""
    m, n = np.shape(C)
    return _solve(C, A_eq=_col_sums(m, n), b_eq=np.asarray(v, np.float64))


def block_ot_lp(C, u, v, groups):
    """Block-constrained OT (Eq. 19): balanced marginals and P_qj = 0 unless
    target j lies in group q.  C rows are the K prototypes, in group order."""
    m, n = np.shape(C)
    groups = np.asarray(groups)
    zero = np.array([[groups[j] != q for j in range(n)] for q in range(m)])
    A = np.vstack([_row_sums(m, n), _col_sums(m, n)])
    return _solve(C, A_eq=A, b_eq=np.concatenate([u, v]), zero_mask=zero)

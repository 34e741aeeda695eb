"""FST capacity, float64 (Sec. 3.4, Eq. 9-10).  Test infrastructure only.

r_j is the mean alpha-weighted FST discrepancy of token t_j to its n nearest
tokens in 3D (Eq. 9); v_j = phi(r_j) / sum_l phi(r_l) (Eq. 10).

Readings of what the paper leaves open:
  * N_n(j) holds the n tokens nearest to t_j other than t_j itself, in the
    (squared distance, index) order of the local greedy's tables (a token's
    discrepancy to itself is 0 and would only dilute its score).
  * d_f, d_x and d_tau are the discrepancies of the cost (Eq. 7) with t_j as
    the first argument: d_f = 1 - cos clamped to [0, 2] (cos = 0 for a
    zero-norm feature), d_x the Euclidean distance, d_tau(t_j, t_k) =
    ReLU(tau_j - tau_k).
  * "normalised within the current sample": each discrepancy is divided by
    its maximum over the N * n (j, k) pairs the scores use (0 when that
    maximum is 0).  Eq. 9 puts no phi_kappa on the spatial term.
  * phi of Eq. 10 is the identity; when every r_j is 0, v is uniform.
"""
from __future__ import annotations

import numpy as np

from . import knn


def neighbours_excluding_self(pos, n_nb: int) -> np.ndarray:
    """[N, n_nb] table: row j lists the n_nb tokens nearest to j other than j,
    by (squared distance, index)."""
    N = np.asarray(pos).shape[0]
    if not 1 <= n_nb <= N - 1:
        raise ValueError("need 1 <= n <= N - 1")
    out = np.empty((N, n_nb), np.int64)
    for lo in range(0, N, 1024):            # row blocks only bound the memory of the distance table
        rows = np.arange(lo, min(N, lo + 1024))
        table = knn.knn_ref(pos, n_nb + 1, rows=rows)
        for i, j in enumerate(rows):
            out[j] = [k for k in table[i] if k != j][:n_nb]
    return out


def pair_discrepancies(F, X, tau, js, ks, block: int = 4096):
    """(d_f, d_x, d_tau) for the ordered pairs (js[i], ks[i]), float64."""
    F = np.asarray(F, np.float64)
    X = np.asarray(X, np.float32).astype(np.float64)
    tau = np.asarray(tau, np.float64)
    js = np.asarray(js, np.int64)
    ks = np.asarray(ks, np.int64)
    norms = np.sqrt(np.sum(F * F, axis=1))
    d_f = np.empty(js.size)
    for lo in range(0, js.size, block):
        a, b = js[lo:lo + block], ks[lo:lo + block]
        dot = np.einsum("ij,ij->i", F[a], F[b])
        den = norms[a] * norms[b]
        cos = np.divide(dot, den, out=np.zeros_like(dot), where=den > 0)
        d_f[lo:lo + block] = np.clip(1.0 - cos, 0.0, 2.0)
    diff = X[js] - X[ks]
    d_x = np.sqrt(np.sum(diff * diff, axis=1))
    d_t = np.maximum(tau[js] - tau[ks], 0.0)
    return d_f, d_x, d_t


def capacity_ref(F, X, tau, n_nb: int, alpha=(1.0, 1.0, 1.0), neighbours=None):
    """FST capacity of every token (Eq. 9-10 under the readings above).

    Returns dict(v, r, neighbours, maxima): the capacity [N] (sums to 1), the
    scores r [N], the neighbour table [N, n_nb] and (M_f, M_x, M_tau)."""
    N = np.asarray(X).shape[0]
    nb = neighbours_excluding_self(X, n_nb) if neighbours is None else np.asarray(neighbours, np.int64)
    js = np.repeat(np.arange(N), n_nb)
    ks = nb.ravel()
    d_f, d_x, d_t = pair_discrepancies(F, X, tau, js, ks)
    maxima = (float(d_f.max()), float(d_x.max()), float(d_t.max()))

    def norm(d, m):
        return d / m if m > 0 else np.zeros_like(d)

    a_f, a_x, a_t = (float(a) for a in alpha)
    s = a_f * norm(d_f, maxima[0]) + a_x * norm(d_x, maxima[1]) + a_t * norm(d_t, maxima[2])
    r = s.reshape(N, n_nb).mean(axis=1)
    total = r.sum()
    v = r / total if total > 0 else np.full(N, 1.0 / N)
    return dict(v=v, r=r, neighbours=nb, maxima=maxima)

"""FST transport cost, float64 (Sec. 3.3, Eq. 7-8).  Test infrastructure only.

Orientation: C[s, t] is the cost of covering target token t with retained
(source) token s, i.e. row = source, column = target, as in Eq. 8 where
C_ij pairs a retained s_i with an original t_j.  The GPU library stores the
transpose (target-major); ``target_major`` converts.

Readings:
  * cos of a zero-norm feature with anything is 0; d_f is clamped to [0, 2]
    and d_f(t, t) is exactly 0.
  * "min-max normalised within the current sample" (Eq. 8): the maximum is
    taken over all N^2 ordered token pairs of the scene, the diagonal
    included.  Every discrepancy is >= 0 and d(t, t) = 0, so the minimum is
    exactly 0 and the normalised value is d / M (0 when M = 0).
  * kappa = 0 denotes the kappa -> 0 limit of phi_kappa, the identity.
  * d_tau(s, t) = ReLU(tau_s - tau_t) with tau the frame index: a later
    source covering an earlier target is penalised (Eq. 7).
"""
from __future__ import annotations

import numpy as np


def widen_features(feats, dtype: str) -> np.ndarray:
    """Stored features as float64.  bfloat16 arrives as uint16 bit patterns;
    widening is exact."""
    if dtype == "bf16":
        bits = np.asarray(feats, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
        return bits.view(np.float32).astype(np.float64)
    if dtype == "f32":
        return np.asarray(feats, dtype=np.float32).astype(np.float64)
    raise ValueError(dtype)


def _rows(n, rows):
    return np.arange(n) if rows is None else np.asarray(rows, dtype=np.int64)


def feature_discrepancy(F: np.ndarray, rows=None) -> np.ndarray:
    """d_f(s, t) = 1 - cos(f_s, f_t) for sources s in ``rows``, all targets t (Eq. 7)."""
    F = np.asarray(F, np.float64)
    r = _rows(F.shape[0], rows)
    norms = np.sqrt(np.sum(F * F, axis=1))
    gram = F[r] @ F.T
    denom = norms[r][:, None] * norms[None, :]
    cos = np.divide(gram, denom, out=np.zeros_like(gram), where=denom > 0)
    d = np.clip(1.0 - cos, 0.0, 2.0)
    d[np.arange(r.size), r] = 0.0
    return d


def spatial_discrepancy(X: np.ndarray, rows=None) -> np.ndarray:
    """d_x(s, t) = ||x_s - x_t||_2 (Eq. 7)."""
    X = np.asarray(X, np.float64)
    r = _rows(X.shape[0], rows)
    diff = X[r][:, None, :] - X[None, :, :]
    return np.sqrt(np.sum(diff * diff, axis=2))


def temporal_discrepancy(tau: np.ndarray, rows=None) -> np.ndarray:
    """d_tau(s, t) = ReLU(tau_s - tau_t) (Eq. 7)."""
    tau = np.asarray(tau, np.float64)
    r = _rows(tau.shape[0], rows)
    return np.maximum(tau[r][:, None] - tau[None, :], 0.0)


def sample_maxima(F, X, tau, block: int = 1024):
    """(M_f, M_x, M_tau): each discrepancy's maximum over all ordered pairs of
    the scene (the normaliser of Eq. 8).  Sources are visited in chunks of
    ``block`` rows only to bound memory; a maximum does not depend on order."""
    n = np.asarray(X).shape[0]
    m_f = m_x = m_t = 0.0
    for lo in range(0, n, block):
        r = np.arange(lo, min(n, lo + block))
        m_f = max(m_f, float(feature_discrepancy(F, r).max()))
        m_x = max(m_x, float(spatial_discrepancy(X, r).max()))
        m_t = max(m_t, float(temporal_discrepancy(tau, r).max()))
    return m_f, m_x, m_t


def phi(z, kappa: float):
    """phi_kappa(z) = log(1 + kappa z) / log(1 + kappa) (Eq. 8); kappa = 0 is the identity limit."""
    z = np.asarray(z, np.float64)
    if kappa == 0.0:
        return z
    return np.log1p(kappa * z) / np.log1p(kappa)


def _normalise(d, m):
    return d / m if m > 0 else np.zeros_like(d)


def fst_cost_ref(F, X, tau, weights=(1.0, 1.0, 1.0), kappa: float = 10.0, rows=None,
                 maxima=None):
    """FST cost C[s, t] = lam_f d_f/M_f + lam_x phi(d_x/M_x) + lam_tau d_tau/M_tau (Eq. 8)
    for sources s in ``rows`` (default: all) and every target t.

    Returns (C, (M_f, M_x, M_tau)).  ``maxima`` may pass normalisers already
    computed by ``sample_maxima`` for the same scene."""
    lam_f, lam_x, lam_t = (float(w) for w in weights)
    if maxima is None:
        maxima = sample_maxima(F, X, tau)
    m_f, m_x, m_t = maxima
    C = lam_f * _normalise(feature_discrepancy(F, rows), m_f)
    C = C + lam_x * phi(_normalise(spatial_discrepancy(X, rows), m_x), kappa)
    C = C + lam_t * _normalise(temporal_discrepancy(tau, rows), m_t)
    return C, maxima


def target_major(C: np.ndarray) -> np.ndarray:
    """The library's storage order: element [t, s] holds C(s, t)."""
    return np.ascontiguousarray(np.asarray(C).T)

"""CoverPrune-Lite, float64 and exact integers (Sec. 4, Eq. 17-20).
Test infrastructure only.

Steps, in the paper's order:
  1. order all tokens along a Morton (Z-order) curve of their 3D positions;
  2. walk that order accumulating capacity and cut K contiguous groups of
     about 1/K capacity each (Eq. 17);
  3. in every group pick the token whose capacity-weighted cost to the
     group is smallest (Eq. 18).
The objective reported is the block-plan transport cost of Eq. 20 with the
closed-form coupling P_qj = v_j that the paper derives for exact 1/K groups.

Readings (the paper fixes none of these):
  * Morton quantisation: origin at the per-axis minimum of the positions,
    isotropic step h / 2^8 (8 sub-voxel bits, so a voxel of edge h is a
    contiguous run of the order), q = floor((x - min) * (2^8 / h)) in
    float64 clamped to [0, 2^21 - 1]; the key interleaves x into bit 3i,
    y into 3i+1, z into 3i+2; ties in the key go to the smaller index.
    A token's voxel is q >> 8 per axis.
  * Grouping (Eq. 17) with cumulative thresholds in exact integers:
    V_j = floor(v_j * 2^40), W = sum V; before token p of the order the
    running group q is closed when K * (mass of tokens before p) reaches
    (q + 1) * W, and it is also closed when the tokens left equal the groups
    left, so that exactly K non-empty contiguous groups result.
  * Locality: a same-group pair whose voxels differ by more than one cell on
    any axis (not among the 27 neighbouring cells) is not evaluated and
    costs c0 = lam_f + lam_x + lam_tau.
  * Normalisation: Lite never forms the full pair set, so the maxima of
    Eq. 8 are taken over the evaluated pairs: ordered same-group,
    27-adjacent pairs, the diagonal included.  A zero maximum zeroes its term.
  * The sum of Eq. 18 includes t itself (cost 0); ties go to the smaller
    token index.
"""
from __future__ import annotations

import math

import numpy as np

from . import fst as _fst

SUB_BITS = 8
AXIS_BITS = 21
CAP_BITS = 40


def quantise(X, h: float):
    """Integer grid coordinates q [N, 3] (Python ints) for voxel size h."""
    X = np.asarray(X, np.float32)
    origin = [float(X[:, a].min()) for a in range(3)]
    scale = float(2 ** SUB_BITS) / float(np.float32(h))
    top = 2 ** AXIS_BITS - 1
    q = []
    for i in range(X.shape[0]):
        row = []
        for a in range(3):
            val = math.floor((float(X[i, a]) - origin[a]) * scale)
            row.append(min(max(val, 0), top))
        q.append(row)
    return q


def morton_key(qx: int, qy: int, qz: int) -> int:
    """Interleave the bits of three coordinates: x -> 3i, y -> 3i+1, z -> 3i+2."""
    key = 0
    for i in range(AXIS_BITS):
        key |= ((qx >> i) & 1) << (3 * i)
        key |= ((qy >> i) & 1) << (3 * i + 1)
        key |= ((qz >> i) & 1) << (3 * i + 2)
    return key


def morton_order(keys):
    """Token indices sorted by (key, index)."""
    return sorted(range(len(keys)), key=lambda i: (keys[i], i))


def capacity_groups(v_in_order, K: int):
    """Group id of each position of the order (Eq. 17 reading above)."""
    n = len(v_in_order)
    if not 1 <= K <= n:
        raise ValueError("need 1 <= K <= N")
    V = [math.floor(float(x) * 2 ** CAP_BITS) for x in v_in_order]
    W = sum(V)
    groups = [0] * n
    q = 0
    before = 0
    for p in range(1, n):
        before += V[p - 1]
        reached = K * before >= (q + 1) * W
        forced = (n - p) == (K - 1 - q)
        if q < K - 1 and (reached or forced):
            q += 1
        groups[p] = q
    return groups


def lite_ref(F, X, tau, v, K: int, weights=(1.0, 1.0, 1.0), kappa: float = 10.0,
             h: float = 0.25):
    """CoverPrune-Lite selection.  F float64 [N, D], X [N, 3], tau [N], v [N].

    Returns dict(selected [K] token of each group q, group [N] group of each
    token, objective, order, keys, maxima (M_f, M_x, M_tau), cost [N] the
    within-group weighted cost of each token)."""
    F = np.asarray(F, np.float64)
    X32 = np.asarray(X, np.float32)
    tau = np.asarray(tau)
    v = np.asarray(v, np.float32)
    n = X32.shape[0]
    lam_f, lam_x, lam_t = (float(w) for w in weights)
    c0 = lam_f + lam_x + lam_t

    q = quantise(X32, h)
    keys = [morton_key(*row) for row in q]
    order = morton_order(keys)
    gpos = capacity_groups([v[i] for i in order], K)
    group = np.empty(n, np.int64)
    members = [[] for _ in range(K)]
    for p, i in enumerate(order):
        group[i] = gpos[p]
        members[gpos[p]].append(i)
    voxel = np.array([[c >> SUB_BITS for c in row] for row in q], np.int64)

    # Pass 1: raw discrepancies of the evaluated pairs and their maxima.
    blocks = []
    m_f = m_x = m_t = 0.0
    for mem in members:
        idx = np.array(mem, np.int64)
        adj = np.all(np.abs(voxel[idx][:, None, :] - voxel[idx][None, :, :]) <= 1, axis=2)
        d_f = _fst.feature_discrepancy(F[idx])
        d_x = _fst.spatial_discrepancy(X32[idx])
        d_t = _fst.temporal_discrepancy(tau[idx])
        m_f = max(m_f, float(d_f[adj].max()))
        m_x = max(m_x, float(d_x[adj].max()))
        m_t = max(m_t, float(d_t[adj].max()))
        blocks.append((idx, adj, d_f, d_x, d_t))

    # Pass 2: FST cost of the evaluated pairs, c0 elsewhere; per-group argmin (Eq. 18).
    def norm(d, m):
        return d / m if m > 0 else np.zeros_like(d)

    cost = np.zeros(n)
    selected = np.empty(K, np.int64)
    objective = 0.0
    for qi, (idx, adj, d_f, d_x, d_t) in enumerate(blocks):
        C = lam_f * norm(d_f, m_f) + lam_x * _fst.phi(norm(d_x, m_x), kappa) + lam_t * norm(d_t, m_t)
        C = np.where(adj, C, c0)
        w = v[idx].astype(np.float64)
        c = C @ w                         # c[t] = sum_j v_j C(t, j)
        cost[idx] = c
        best = min(range(idx.size), key=lambda a: (c[a], idx[a]))
        selected[qi] = idx[best]
        objective += float(c[best])
    return dict(selected=selected, group=group, objective=objective,
                order=np.array(order, np.int64), keys=np.array(keys, np.uint64),
                maxima=(m_f, m_x, m_t), cost=cost, voxel=voxel)

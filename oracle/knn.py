"""Nearest neighbours in 3D for the local greedy (Sec. 3.5, Eq. 13), float64.
Test infrastructure only.

M_g(t) = NN_g(t; T): the g target tokens nearest to t in 3D space.  Reading
of what the paper leaves open: distances are Euclidean on the token
positions; t itself belongs to its own neighbourhood (distance 0); equal
distances are broken by the smaller token index; comparisons use the squared
distance formed in float64 from the float32 positions as (dx^2 + dy^2) + dz^2
(no fused multiply-add), which orders exactly like the distance.
"""
from __future__ import annotations

import numpy as np


def sq_dist_rows(pos, rows=None):
    """Squared distances [len(rows), N] from the given rows to every token."""
    p = np.asarray(pos, np.float32).astype(np.float64)
    r = p if rows is None else p[np.asarray(rows)]
    dx = r[:, 0][:, None] - p[:, 0][None, :]
    dy = r[:, 1][:, None] - p[:, 1][None, :]
    dz = r[:, 2][:, None] - p[:, 2][None, :]
    return (dx * dx + dy * dy) + dz * dz


def knn_ref(pos, g: int, rows=None):
    """Table [len(rows), g] of M_g(t) for each t in rows (all tokens when
    rows is None): the g nearest tokens ordered by (squared distance, index)."""
    n = np.asarray(pos).shape[0]
    if not 1 <= g <= n:
        raise ValueError("need 1 <= g <= N")
    d2 = sq_dist_rows(pos, rows)
    idx = np.arange(n)
    out = np.empty((d2.shape[0], g), np.int64)
    for a in range(d2.shape[0]):
        order = np.lexsort((idx, d2[a]))      # primary key: distance, then index
        out[a] = order[:g]
    return out

"""Coverage loss and Spatial-Guided Greedy Selection, float64 (Sec. 3.5,
Eq. 11-16).  Test infrastructure only.

Reading of the per-step transport solve (Eq. 11-14).  The paper leaves the
source capacities, epsilon and the solver of the per-step semi-relaxed
problem open.  In the limit epsilon -> 0 with the retained tokens' masses
left free, every target's capacity v_j flows whole to its cheapest retained
token, or stays uncovered at cost c0 (the largest value the cost can take,
lam_f + lam_x + lam_tau).  The set function this induces,

    L(S) = sum_j v_j * min(c0, min_{s in S} C(s, j)),

is the relaxed coverage loss; L(empty) - L(S) is monotone submodular, which
is what licenses the greedy the paper invokes.  The residual of Eq. 14 is
then carried by the per-target best cost b_j = min(c0, min_{s in S} C(s, j)),
and the residual-weighted marginal cost minimised in Eq. 15 is the change of
L from adding candidate c:

    L(S + c) - L(S) = -gain(c),   gain(c) = sum_{j in M_g(c)} v_j * max(0, b_j - C(c, j)).

With g = N (every target is a neighbour) this is exact greedy on L.  Ties in
the gain go to the smallest token index; the already selected tokens are not
candidates (Eq. 15); a step with zero gain still selects, so |S| = K.
"""
from __future__ import annotations

import heapq
import itertools
import math

import numpy as np


def coverage_loss(C, v, S, c0: float) -> float:
    """L(S) = sum_j v_j min(c0, min_{s in S} C(s, j))."""
    C = np.asarray(C, np.float64)
    v = np.asarray(v, np.float64)
    S = list(S)
    if not S:
        return float(np.sum(v) * c0)
    best = np.minimum(c0, C[S].min(axis=0))
    return float(np.sum(v * best))


def sgs_ref(C, v, K: int, c0: float, neighbours=None):
    """Greedy selection of K tokens (Eq. 15-16 under the reading above).

    C: source-major costs [N, N] (C[s, t]).  v: target capacities [N].
    neighbours: optional [N, g] integer table; row c lists the targets M_g(c)
    whose gain candidate c may claim (Eq. 13).  None means all N targets.

    Returns dict(selected, gain, objective, assign): selected tokens in greedy
    order; the gain of each step; L(S) after each step; and for every target
    the retained token that covers it most cheaply (-1 while it is uncovered).
    """
    C = np.asarray(C, np.float64)
    v = np.asarray(v, np.float64)
    n = C.shape[0]
    if not 1 <= K <= n:
        raise ValueError("need 1 <= K <= N")
    if neighbours is not None:
        local = np.zeros((n, n), bool)
        nb = np.asarray(neighbours)
        local[np.repeat(np.arange(n), nb.shape[1]), nb.ravel()] = True
    b = np.full(n, float(c0))
    chosen = np.zeros(n, bool)
    assign = np.full(n, -1, np.int64)
    selected, gains, objectives = [], [], []
    for _ in range(K):
        contrib = v[None, :] * np.maximum(0.0, b[None, :] - C)
        if neighbours is not None:
            contrib = np.where(local, contrib, 0.0)
        gain = contrib.sum(axis=1)
        gain[chosen] = -np.inf
        t = int(np.argmax(gain))            # first maximum: smallest index on ties
        chosen[t] = True
        better = C[t] < b
        assign[better] = t
        b = np.minimum(b, C[t])
        selected.append(t)
        gains.append(float(gain[t]))
        objectives.append(float(np.sum(v * b)))
    return dict(selected=np.array(selected, np.int64), gain=np.array(gains),
                objective=np.array(objectives), assign=assign, best=b)


def lazy_greedy_ref(C, v, K: int, c0: float):
    """Minoux's lazy greedy on the same set function: an independent route to
    the same selections (exact greedy, since gains only shrink as S grows).
    Each candidate's gain is evaluated on its own, with math.fsum."""
    C = np.asarray(C, np.float64)
    v = np.asarray(v, np.float64)
    n = C.shape[0]
    b = np.full(n, float(c0))

    def gain_of(c):
        return math.fsum((v * np.maximum(0.0, b - C[c])).tolist())

    heap = [(-gain_of(c), c, 0) for c in range(n)]
    heapq.heapify(heap)
    selected = []
    for step in range(K):
        while True:
            neg, c, stamp = heapq.heappop(heap)
            if stamp == step:
                break
            heapq.heappush(heap, (-gain_of(c), c, step))
        selected.append(c)
        b = np.minimum(b, C[c])
    return np.array(selected, np.int64)


def enumerate_ref(C, v, K: int, c0: float):
    """Exhaustive minimiser of L(S) over all |S| = K (Eq. 6 under the relaxed
    loss).  Returns (best loss, best set as a sorted tuple).  Tiny N only."""
    n = np.asarray(C).shape[0]
    best = (math.inf, None)
    for S in itertools.combinations(range(n), K):
        val = coverage_loss(C, v, S, c0)
        if val < best[0]:
            best = (val, S)
    return best

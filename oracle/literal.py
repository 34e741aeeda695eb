"""The greedy step solved as the paper writes it, float64 (Sec. 3.5,
Eq. 11-15).  Test infrastructure only.

Each step solves the entropic semi-relaxed transport of Eq. 12 between the
tokens retained so far and all targets, takes the residual capacity of
Eq. 14, and picks the token with the smallest residual-weighted cost
(Eq. 15).

Readings of what the paper leaves open:
  * source masses: u_i = 1/K for every retained token (K the budget), so at
    step l the sources carry l/K of the unit target mass and the residual is
    not zero (normalising u over S_l would make the relaxation tight and r = 0);
  * Eq. 12 is min <P, C_S> - eps H(P) subject to P 1 = u, P^T 1 <= v, solved
    by alternating scalings P = diag(a) E diag(b) with E = exp(-C_S / eps):
    a <- u / (E b), then b <- min(1, v / (E^T a)) (b_j = 1 where E^T a is 0),
    starting from b = 1 at every step, for a fixed number of rounds; eps and
    the round count are inputs;
  * residual r = [v - P^T 1]_+ with P^T 1 = b * (E^T a) after the last round;
    with no token retained, r = v;
  * Eq. 15 with M_g(t) = every target (g = N): the next token minimises
    sum_j r_j C(t, j) over the unselected tokens, ties to the smaller index
    (for g < N a covered neighbourhood scores 0 and the literal rule is
    degenerate, so only g = N is taken);
  * objective: the transport cost <P, C_S> of the plan solved for the final
    set (l = K: u sums to 1 like v, so the plan is the balanced one).
"""
from __future__ import annotations

import numpy as np


def sot_scaling(C_S, u, v, eps: float, rounds: int):
    """Scalings (a, b) and kernel E of the entropic semi-relaxed transport
    between sources with masses u (rows of C_S) and targets with capacities v.
    The plan is P = a[:, None] * E * b[None, :]."""
    C_S = np.asarray(C_S, np.float64)
    u = np.asarray(u, np.float64)
    v = np.asarray(v, np.float64)
    E = np.exp(-C_S / eps)
    b = np.ones(C_S.shape[1])
    a = np.zeros(C_S.shape[0])
    for _ in range(rounds):
        a = u / (E @ b)
        t = E.T @ a
        b = np.where(t > 0, np.minimum(1.0, np.divide(v, t, out=np.ones_like(t), where=t > 0)), 1.0)
    return a, b, E


def literal_sgs_ref(C, v, K: int, eps: float, rounds: int, follow=None, steps=None):
    """K steps of the literal greedy (readings above) on the source-major cost C.

    follow: optional picks to take instead of the oracle's own (a replay of
    another trajectory); the oracle's scores are still reported for them.
    steps: optionally stop after that many steps (the sources keep mass 1/K);
    the objective is then None.

    Returns dict(selected, score, best, residual, objective): the picks; the
    score sum_j r_j C(t, j) of each pick; the smallest score among the
    unselected tokens at each step; the residual mass sum_j r_j before each
    pick; and the final plan's transport cost."""
    C = np.asarray(C, np.float64)
    v = np.asarray(v, np.float64)
    n = C.shape[0]
    if not 1 <= K <= n:
        raise ValueError("need 1 <= K <= N")
    chosen = np.zeros(n, bool)
    S, scores, bests, residual = [], [], [], []
    for step in range(K if steps is None else min(K, steps)):
        if S:
            a, b, E = sot_scaling(C[S], np.full(len(S), 1.0 / K), v, eps, rounds)
            r = np.maximum(v - b * (E.T @ a), 0.0)
        else:
            r = v.copy()
        score = C @ r
        score[chosen] = np.inf
        best = int(np.argmin(score))        # first minimum: smallest index on ties
        t = best if follow is None else int(follow[step])
        if chosen[t]:
            raise ValueError(f"step {step}: token {t} already selected")
        scores.append(float(score[t]))
        bests.append(float(score[best]))
        residual.append(float(r.sum()))
        chosen[t] = True
        S.append(t)
    objective = None
    if len(S) == K:
        a, b, E = sot_scaling(C[S], np.full(K, 1.0 / K), v, eps, rounds)
        P = a[:, None] * E * b[None, :]
        objective = float(np.sum(P * C[S]))
    return dict(selected=np.array(S, np.int64), score=np.array(scores), best=np.array(bests),
                residual=np.array(residual), objective=objective)

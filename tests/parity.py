"""Comparison helpers for the GPU parity tests.  Expected values always come
from the oracle; GPU outputs are only ever the thing being checked."""
from __future__ import annotations

import functools
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
from threadpoolctl import threadpool_limits

from oracle import capacity, fst, knn, lite, sgs
from scenes import make_scene, subscene

# Cost tolerance: bf16 inputs with float32 accumulation against float64.
COST_RTOL = 1e-3
COST_ATOL = 1e-5
# Gains within this relative distance of the best count as ties.
TIE_RTOL = 1e-6


@functools.lru_cache(maxsize=8)
def _scene(cfg, seed):
    return make_scene(cfg, seed)


def sample_scene(cfg, n, seed, salt=0):
    """``n`` random tokens (sorted) of a generated scene; the whole scene for
    n = None.  Always a fresh copy, so callers may modify it."""
    s = _scene(cfg, seed)
    if n is None or n >= s.n:
        return subscene(s, np.arange(s.n), renormalise=False)
    idx = np.sort(np.random.default_rng(salt + seed).choice(s.n, size=n, replace=False))
    return subscene(s, idx)


def oracle_neighbours_excluding_self(pos, n_nb, block=512):
    """``capacity.neighbours_excluding_self`` built from row blocks of the
    oracle's kNN table on a thread pool (the same table: each row's n_nb + 1
    nearest tokens by (distance, index), the row's own token dropped)."""
    n = np.asarray(pos).shape[0]
    out = np.empty((n, n_nb), np.int64)

    def rows(lo):
        r = np.arange(lo, min(n, lo + block))
        table = knn.knn_ref(pos, n_nb + 1, rows=r)
        for i, j in enumerate(r):
            out[j] = [k for k in table[i] if k != j][:n_nb]

    with ThreadPoolExecutor(_workers()) as pool:
        list(pool.map(rows, range(0, n, block)))
    return out


def workload_scene(cfg, seed):
    """A whole workload scene with the workload's own capacities: the
    generator's recipe, or the oracle's FST capacity (Eq. 9-10) where the
    workload names it.  Inputs of both the library and the oracle."""
    s = make_scene(cfg, seed)
    nn = s.config.fst_capacity_nn
    if nn:
        F = fst.widen_features(s.feats, s.dtype)
        nb = oracle_neighbours_excluding_self(s.pos, nn)
        s.capacity = capacity.capacity_ref(F, s.pos, s.frame, nn, neighbours=nb)["v"].astype(np.float32)
    return s


def oracle_cost(scene, weights=(1.0, 1.0, 1.0), kappa=10.0, rows=None, maxima=None):
    F = fst.widen_features(scene.feats, scene.dtype)
    return fst.fst_cost_ref(F, scene.pos, scene.frame, weights=weights, kappa=kappa, rows=rows,
                            maxima=maxima)


def oracle_cost_f32_target_major(scene, weights=(1.0, 1.0, 1.0), kappa=10.0, block=2048):
    """The oracle's full cost rounded to float32, target-major, built in row
    blocks so that large scenes fit in memory."""
    F = fst.widen_features(scene.feats, scene.dtype)
    maxima = fst.sample_maxima(F, scene.pos, scene.frame, block=block)
    n = scene.n
    out = np.empty((n, n), np.float32)
    for lo in range(0, n, block):
        rows = np.arange(lo, min(n, lo + block))
        C, _ = fst.fst_cost_ref(F, scene.pos, scene.frame, weights=weights, kappa=kappa, rows=rows,
                                maxima=maxima)
        out[:, lo:lo + rows.size] = C.T.astype(np.float32)
    return out, maxima


def _workers():
    return max(1, min(16, os.cpu_count() or 1))


def oracle_cost_full(scene, weights=(1.0, 1.0, 1.0), kappa=10.0, block=256):
    """The oracle's whole cost C[s, t] in float64, source-major, for scenes of
    up to tens of thousands of tokens.  Each row block is one call of the
    oracle on a thread pool (one BLAS thread per call); the normalisers are
    the oracle's discrepancy maxima over every block, exactly what
    ``fst.sample_maxima`` returns (a maximum does not depend on the order)."""
    F = fst.widen_features(scene.feats, scene.dtype)
    n = scene.n
    blocks = [np.arange(lo, min(n, lo + block)) for lo in range(0, n, block)]

    def block_max(r):
        return (float(fst.feature_discrepancy(F, r).max()), float(fst.spatial_discrepancy(scene.pos, r).max()),
                float(fst.temporal_discrepancy(scene.frame, r).max()))

    out = np.empty((n, n), np.float64)

    def block_cost(r):
        C, _ = fst.fst_cost_ref(F, scene.pos, scene.frame, weights=weights, kappa=kappa, rows=r, maxima=maxima)
        out[r[0]:r[-1] + 1] = C

    with threadpool_limits(1), ThreadPoolExecutor(_workers()) as pool:
        parts = list(pool.map(block_max, blocks))
        maxima = tuple(max(p[i] for p in parts) for i in range(3))
        list(pool.map(block_cost, blocks))
    return out, maxima


def assert_cost_close(gpu_tm: np.ndarray, ref_source_major: np.ndarray):
    """gpu_tm[t, s] = C(s, t) against the oracle's C[s, t]."""
    ref_tm = ref_source_major.T
    err = np.abs(gpu_tm.astype(np.float64) - ref_tm)
    bound = COST_RTOL * np.abs(ref_tm) + COST_ATOL
    bad = err > bound
    if bad.any():
        t, s = np.argwhere(bad)[0]
        raise AssertionError(f"{int(bad.sum())} cost entries off; first at target {t}, source {s}: "
                             f"gpu {gpu_tm[t, s]!r} oracle {ref_tm[t, s]!r}; max err {err.max():.3g}")
    return float(err.max())


def replay_greedy(C_src: np.ndarray, v: np.ndarray, c0: float, picks, tie_atol=0.0):
    """Check that ``picks`` is a valid greedy trajectory on the oracle's cost.

    At every step the pick must be unselected and its exact gain (oracle
    arithmetic, on the trajectory so far) within TIE_RTOL * best + tie_atol of
    the best gain.  Returns (steps where the pick was not the oracle's own
    first choice, oracle gains of the picks, oracle objectives)."""
    C = np.asarray(C_src, np.float64)
    v = np.asarray(v, np.float64)
    n = C.shape[0]
    b = np.full(n, float(c0))
    chosen = np.zeros(n, bool)
    ties, gains, objs = [], [], []
    for step, t in enumerate(int(x) for x in picks):
        assert 0 <= t < n and not chosen[t], f"step {step}: pick {t} invalid or repeated"
        g = (v[None, :] * np.maximum(0.0, b[None, :] - C)).sum(axis=1)
        g[chosen] = -np.inf
        best = int(np.argmax(g))
        if t != best:
            slack = TIE_RTOL * abs(g[best]) + tie_atol
            assert g[t] >= g[best] - slack, (f"step {step}: picked {t} with gain {g[t]!r}, "
                                             f"best is {best} with {g[best]!r}")
            ties.append(step)
        chosen[t] = True
        gains.append(g[t])
        b = np.minimum(b, C[t])
        objs.append(float(np.sum(v * b)))
    return ties, np.array(gains), np.array(objs)


def _row_gains(C, rows, v, b):
    """Exact float64 gains sum_j v_j max(0, b_j - C(c, j)) of the source rows
    ``rows`` (an integer array, so indexing copies), the formula of
    ``replay_greedy``."""
    X = np.asarray(C[np.asarray(rows, np.int64)], np.float64)
    if X.base is not None or X.dtype != np.float64:
        X = np.array(X, np.float64)
    np.subtract(b[None, :], X, out=X)
    np.maximum(X, 0.0, out=X)
    X *= v[None, :]
    return X.sum(axis=1)


def _gains(C, rows, v, b, pool, chunk=256):
    rows = np.asarray(rows, np.int64)
    if pool is None or rows.size <= chunk:
        return _row_gains(C, rows, v, b)
    return np.concatenate(list(pool.map(lambda lo: _row_gains(C, rows[lo:lo + chunk], v, b),
                                        range(0, rows.size, chunk))))


def lazy_replay(C, v, c0: float, picks, tie_atol=0.0, alt=None, tie_rtol=TIE_RTOL):
    """``replay_greedy`` for full-size trajectories.

    C is the source-major cost (float32 or float64; C[c, j] = C(c, j)) on
    which the oracle evaluates exact float64 gains along the trajectory
    ``picks``.  Every candidate keeps an upper bound on its gain, the gain it
    had when last evaluated: gains only shrink as targets get covered (the
    coverage function is submodular, Sec. 3.5), so a candidate whose bound is
    below the pick's gain cannot beat or tie the pick, and only the others
    are evaluated again.  The check is therefore the same as evaluating
    every candidate at every step.

    A competitor c beats the pick t if its gain is larger, or equal at a
    smaller index; the pick is accepted when
    gain(t) >= gain(c) - (tie_rtol * gain(c) + tie_atol + delta_t + delta_c)
    for every such c.  ``alt`` is the source-major cost the picks were made
    on, when it is not C (end-to-end runs): then delta_c = sum_j v_j (|b_j -
    b'_j| + |C(c, j) - C'(c, j)|), with b' the best costs under ``alt``, bounds
    how far c's gain under ``alt`` is from its gain under C; otherwise delta = 0.

    Returns (ties, gains, objectives, near): the steps whose pick was not the
    oracle's own choice, the oracle's gains of the picks, L after each step,
    and for each tie step (step, pick, oracle choice, their gains, allowance).
    """
    v = np.asarray(v, np.float64)
    n = C.shape[0]
    b = np.full(n, float(c0))
    b_alt = b.copy() if alt is not None else None
    chosen = np.zeros(n, bool)
    ties, gains, objs, near = [], [], [], []

    def delta(c):
        return float(np.sum(v * (np.abs(b - b_alt) + np.abs(np.asarray(C[c], np.float64) -
                                                             np.asarray(alt[c], np.float64)))))

    with threadpool_limits(1), ThreadPoolExecutor(_workers()) as pool:
        ub = _gains(C, np.arange(n), v, b, pool)
        for step, t in enumerate(int(x) for x in picks):
            assert 0 <= t < n and not chosen[t], f"step {step}: pick {t} invalid or repeated"
            g_t = float(_row_gains(C, [t], v, b)[0])
            cand = np.flatnonzero(ub >= g_t)
            cand = cand[~chosen[cand] & (cand != t)]
            if cand.size:
                g_c = _gains(C, cand, v, b, pool)
                ub[cand] = g_c
                beat = (g_c > g_t) | ((g_c == g_t) & (cand < t))
                if beat.any():
                    comp, g_comp = cand[beat], g_c[beat]
                    slack = tie_rtol * np.abs(g_comp) + tie_atol
                    if alt is not None:
                        d_t = delta(t)
                        slack = slack + d_t + np.array([delta(c) for c in comp])
                    bad = g_t < g_comp - slack
                    if bad.any():
                        c = int(comp[bad][0])
                        raise AssertionError(f"step {step}: picked {t} with gain {g_t!r}, but {c} has "
                                             f"{float(g_comp[bad][0])!r} (allowance {float(slack[bad][0]):.3g})")
                    top = np.flatnonzero(g_comp == g_comp.max())
                    best = int(comp[top].min())
                    ties.append(step)
                    near.append(dict(step=step, pick=t, oracle=best, gain=g_t, oracle_gain=float(g_comp.max()),
                                     allowance=float(np.max(slack))))
            chosen[t] = True
            gains.append(g_t)
            b = np.minimum(b, np.asarray(C[t], np.float64))
            if alt is not None:
                b_alt = np.minimum(b_alt, np.asarray(alt[t], np.float64))
            objs.append(float(np.sum(v * b)))
    return ties, np.array(gains), np.array(objs), near


def replay_greedy_local(C_tm: np.ndarray, v: np.ndarray, c0: float, neighbours, picks, tie_atol=0.0):
    """replay_greedy for the local form (Eq. 13): each candidate's gain runs
    over its neighbour row only, while b is lowered for every target.

    C_tm is target-major (C_tm[j, c] = C(c, j)), so a full-size float32 cost
    fits; gains are formed from the gathered [n, g] band in float64."""
    v = np.asarray(v, np.float64)
    nb = np.asarray(neighbours, np.int64)
    n, g = nb.shape
    rows = np.repeat(np.arange(n), g).reshape(n, g)
    Cg = np.asarray(C_tm[nb, rows], np.float64)            # Cg[c, q] = C(c, nb[c, q])
    vg = v[nb]
    b = np.full(n, float(c0))
    chosen = np.zeros(n, bool)
    ties, gains, objs = [], [], []
    for step, t in enumerate(int(x) for x in picks):
        assert 0 <= t < n and not chosen[t], f"step {step}: pick {t} invalid or repeated"
        gl = (vg * np.maximum(0.0, b[nb] - Cg)).sum(axis=1)
        gl[chosen] = -np.inf
        best = int(np.argmax(gl))
        if t != best:
            slack = TIE_RTOL * abs(gl[best]) + tie_atol
            assert gl[t] >= gl[best] - slack, (f"step {step}: picked {t} with local gain {gl[t]!r}, "
                                               f"best is {best} with {gl[best]!r}")
            ties.append(step)
        chosen[t] = True
        gains.append(gl[t])
        b = np.minimum(b, np.asarray(C_tm[:, t], np.float64))
        objs.append(float(np.sum(v * b)))
    return ties, np.array(gains), np.array(objs)


def check_trajectory_invariants(sel, gain, obj, v, c0, k, n):
    sel = np.asarray(sel)
    assert len(sel) == k and len(set(sel.tolist())) == k
    assert sel.min() >= 0 and sel.max() < n
    v = np.asarray(v, np.float64)
    total = c0 * v.sum()
    # L_k = c0 sum(v) - sum of gains, and L decreases by exactly each gain.
    # The kernel forms b - C in float32 (relative rounding 2^-24 per term).
    assert abs(obj[-1] - (total - gain.sum())) <= 1e-6 * total + 1e-12
    prev = np.concatenate([[total], obj[:-1]])
    assert np.allclose(prev - obj, gain, rtol=1e-6, atol=1e-9 * total)
    # Gains of a monotone submodular function never grow along the greedy.
    assert np.all(np.diff(gain) <= 1e-9 * max(gain[0], 1e-300))


def lite_reference(scene, k, weights=(1.0, 1.0, 1.0), kappa=10.0, h=0.25, capacity=None):
    F = fst.widen_features(scene.feats, scene.dtype)
    v = scene.capacity if capacity is None else capacity
    return lite.lite_ref(F, scene.pos, scene.frame, v, k, weights=weights, kappa=kappa, h=h)


def assert_lite_close(gpu_sel, gpu_group, gpu_obj, ref, gpu_cost, rtol=TIE_RTOL):
    """Lite against the oracle.  Groups bit-exact.  Every token's cost to its
    group (the quantity Eq. 18 minimises) within the cost tolerance of the
    oracle's.  In every group the GPU's prototype costs, by the oracle, at
    most the group's minimum plus rtol of it plus the measured cost errors of
    the two tokens (the GPU picks the least cost by its own values, so
    cost(s) <= cost'(s) + e_s <= cost'(r) + e_s <= cost(r) + e_r + e_s).  The
    objective within the summed allowances.  Returns the number of groups
    whose prototype differs from the oracle's."""
    gpu_group = np.asarray(gpu_group)
    assert np.array_equal(gpu_group, ref["group"]), \
        f"{int((gpu_group != ref['group']).sum())} tokens in a different group"
    cost = ref["cost"]
    gpu_cost = np.asarray(gpu_cost, np.float64)
    err = np.abs(gpu_cost - cost)
    bound = COST_RTOL * np.abs(cost) + COST_ATOL
    assert np.all(err <= bound), f"token cost off by {err.max():.3g} (token {int(np.argmax(err - bound))})"
    gpu_sel = np.asarray(gpu_sel)
    ref_sel = ref["selected"]
    assert np.array_equal(ref["group"][gpu_sel], np.arange(len(gpu_sel))), "prototype outside its group"
    c_gpu = cost[gpu_sel]
    c_ref = cost[ref_sel]
    slack = rtol * np.abs(c_ref) + err[gpu_sel] + err[ref_sel]
    bad = c_gpu > c_ref + slack
    assert not bad.any(), (f"{int(bad.sum())} groups pick a worse prototype; first group "
                           f"{int(np.argmax(bad))}: {c_gpu[bad][0]!r} vs {c_ref[bad][0]!r}")
    assert abs(gpu_obj - float(np.sum(gpu_cost[gpu_sel]))) <= 1e-12 * abs(gpu_obj) + 1e-15
    assert abs(gpu_obj - ref["objective"]) <= float(np.sum(slack + err[gpu_sel])) + 1e-12
    return int((gpu_sel != ref_sel).sum())

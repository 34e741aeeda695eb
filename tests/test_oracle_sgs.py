"""Pins for the oracle's greedy selection (Sec. 3.5, Eq. 11-16): a hand-traced
toy, closed forms, exhaustive search with the greedy guarantee for monotone
submodular maximisation, an independent lazy greedy, and invariants."""
import math

import numpy as np
import pytest

from oracle import fst, sgs
from scenes import make_scene, subscene


def _cost(s, weights=(1.0, 1.0, 1.0), kappa=10.0):
    F = fst.widen_features(s.feats, s.dtype)
    C, _ = fst.fst_cost_ref(F, s.pos, s.frame, weights=weights, kappa=kappa)
    return C


def _sub(n, seed, cfg="n1024_d256_f32"):
    s = make_scene(cfg, seed)
    idx = np.random.default_rng(100 + seed).choice(s.n, size=n, replace=False)
    return subscene(s, np.sort(idx))


def test_toy_trace(toy):
    # Hand trace on the toy cost (c0 = 3, v = 1/4): step 0 gains are
    # (3 - row mean) = 2.051424, 1.938184, 1.638355, 1.584629 -> pick 0.
    # Then b = row 0 of C; gains of 1, 2, 3 are 0.179652, 0.5, 0.375 -> pick 2;
    # then 0.157632 (token 1) vs 0.290944 (token 3) -> pick 3; finally token 1.
    C, _ = fst.fst_cost_ref(toy["F"], toy["X"], toy["tau"])
    out = sgs.sgs_ref(C, toy["v"], 4, 3.0)
    assert list(out["selected"]) == [0, 2, 3, 1]
    assert np.allclose(out["gain"], [2.051424, 0.5, 0.290944, 0.157632], atol=6e-7)
    assert np.allclose(out["objective"], [0.948576, 0.448576, 0.157632, 0.0], atol=6e-7)
    one = sgs.sgs_ref(C, toy["v"], 2, 3.0)
    assert list(one["selected"]) == [0, 2]


def test_single_pick_is_weighted_medoid():
    s = _sub(120, 1)
    C = _cost(s)
    v = s.capacity.astype(np.float64)
    medoid = min(range(len(v)), key=lambda c: (sum(v[j] * C[c, j] for j in range(len(v))), c))
    assert sgs.sgs_ref(C, v, 1, 3.0)["selected"][0] == medoid


def test_full_budget_covers_everything():
    s = _sub(50, 2)
    C = _cost(s)
    out = sgs.sgs_ref(C, s.capacity, 50, 3.0)
    assert sorted(out["selected"]) == list(range(50))
    assert out["objective"][-1] == 0.0


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_trajectory_invariants(seed):
    s = _sub(200, seed, "n4096_d1152")
    C = _cost(s, weights=(1.0, 0.5, 0.8), kappa=4.0)
    c0 = 2.3
    v = s.capacity.astype(np.float64)
    K = 40
    out = sgs.sgs_ref(C, v, K, c0)
    sel = out["selected"]
    assert len(set(sel.tolist())) == K
    # Telescoping: L_K = c0 * sum(v) - sum of gains.
    assert out["objective"][-1] == pytest.approx(c0 * v.sum() - out["gain"].sum(), rel=1e-12)
    # Submodularity: the gains of successive picks never grow; the loss never grows.
    assert np.all(np.diff(out["gain"]) <= 1e-15)
    assert np.all(np.diff(out["objective"]) <= 1e-15)
    # The implied plan P[assign(j), j] = v_j moves every covered target's whole
    # capacity to a retained token, at that token's cost, and reproduces L.
    a = out["assign"]
    assert set(a[a >= 0].tolist()) <= set(sel.tolist())
    per_target = np.where(a >= 0, C[np.maximum(a, 0), np.arange(len(v))], c0)
    assert np.allclose(per_target, np.minimum(c0, C[sel].min(axis=0)))
    assert np.sum(v * per_target) == pytest.approx(out["objective"][-1], rel=1e-12)
    assert sgs.coverage_loss(C, v, sel, c0) == pytest.approx(out["objective"][-1], rel=1e-12)


@pytest.mark.parametrize("seed", range(12))
def test_exhaustive_search_bound(seed):
    # Greedy on a monotone submodular function reaches at least (1 - 1/e) of
    # the best improvement over the empty set (Nemhauser, Wolsey, Fisher 1978).
    rng = np.random.default_rng(seed)
    n = int(rng.integers(6, 13))
    K = int(rng.integers(1, 5))
    s = _sub(n, seed)
    C = _cost(s)
    v = s.capacity.astype(np.float64)
    c0 = 3.0
    base = c0 * v.sum()
    best_loss, best_set = sgs.enumerate_ref(C, v, K, c0)
    out = sgs.sgs_ref(C, v, K, c0)
    greedy_loss = out["objective"][-1]
    assert greedy_loss >= best_loss - 1e-12
    assert base - greedy_loss >= (1 - 1 / math.e) * (base - best_loss) - 1e-12
    if K == 1:
        assert tuple(out["selected"]) == best_set


@pytest.mark.parametrize("seed", [0, 1])
def test_lazy_greedy_agrees(seed):
    s = _sub(150, seed, "n4096_d1152")
    C = _cost(s)
    out = sgs.sgs_ref(C, s.capacity, 30, 3.0)
    lazy = sgs.lazy_greedy_ref(C, s.capacity, 30, 3.0)
    assert list(out["selected"]) == list(lazy)


def test_all_neighbours_equals_dense():
    s = _sub(80, 4)
    C = _cost(s)
    nb = np.tile(np.arange(80), (80, 1))
    a = sgs.sgs_ref(C, s.capacity, 12, 3.0)
    b = sgs.sgs_ref(C, s.capacity, 12, 3.0, neighbours=nb)
    assert list(a["selected"]) == list(b["selected"])


def test_local_neighbourhood_restricts_gain():
    # With g = 1 each candidate can only claim itself, so the first pick is the
    # token with the largest v_j * (c0 - C(j, j)) = c0 * v_j.
    s = _sub(60, 5)
    C = _cost(s)
    v = s.capacity.astype(np.float64)
    nb = np.arange(60)[:, None]
    out = sgs.sgs_ref(C, v, 1, 3.0, neighbours=nb)
    assert out["selected"][0] == int(np.argmax(v))


def test_local_gains_bounded_by_dense_gains():
    # A neighbourhood only drops nonnegative terms: at every step of the local
    # trajectory the pick's local gain is at most its gain over all targets.
    from oracle import knn
    s = _sub(90, 6)
    C = _cost(s)
    v = s.capacity.astype(np.float64)
    nb = knn.knn_ref(s.pos, 7)
    out = sgs.sgs_ref(C, v, 15, 3.0, neighbours=nb)
    b = np.full(90, 3.0)
    for t, g in zip(out["selected"], out["gain"]):
        full = float(np.sum(v * np.maximum(0.0, b - C[t])))
        assert g <= full + 1e-15
        b = np.minimum(b, C[t])
    # L(S) still telescopes over the picks' full gains.
    assert out["objective"][-1] == pytest.approx(float(np.sum(v * b)), rel=1e-12)


def test_local_pick_lowers_best_cost_beyond_its_neighbourhood():
    # Three tokens on a line; each candidate sees only itself (g = 1), but the
    # residual of the transport over all targets (Eq. 14) drops everywhere.
    C = np.array([[0.0, 0.5, 2.0],
                  [0.5, 0.0, 1.0],
                  [2.0, 1.0, 0.0]])
    v = np.array([0.5, 0.3, 0.2])
    nb = np.arange(3)[:, None]
    out = sgs.sgs_ref(C, v, 2, 3.0, neighbours=nb)
    # step 0: local gains are c0 v_c = 1.5, 0.9, 0.6 -> token 0
    assert out["selected"][0] == 0 and out["gain"][0] == pytest.approx(1.5)
    # b after step 0 = min(c0, C[0]) = [0, 0.5, 2.0]; step 1 local gains:
    # token 1: 0.3 (0.5 - 0) = 0.15, token 2: 0.2 (2.0 - 0) = 0.4 -> token 2
    assert out["selected"][1] == 2 and out["gain"][1] == pytest.approx(0.4)
    assert out["objective"][1] == pytest.approx(0.3 * 0.5)


def test_local_replay_agrees_with_local_oracle():
    # The gather-form replay used against GPU trajectories accepts the oracle's
    # own local trajectory with no ties and the same gains and objectives, and
    # rejects a trajectory that swaps a clearly better pick for a worse one.
    from oracle import knn
    from tests import parity
    rng = np.random.default_rng(31)
    n, g, K = 60, 8, 15
    pos = rng.standard_normal((n, 3)).astype(np.float32)
    C = rng.uniform(0.0, 3.0, (n, n))
    np.fill_diagonal(C, 0.0)
    v = rng.uniform(0.5, 1.5, n)
    v /= v.sum()
    nb = knn.knn_ref(pos, g)
    ref = sgs.sgs_ref(C, v, K, 3.0, neighbours=nb)
    ties, gains, objs = parity.replay_greedy_local(np.ascontiguousarray(C.T), v, 3.0, nb, ref["selected"])
    assert ties == []
    assert np.allclose(gains, ref["gain"], rtol=1e-14, atol=0.0)
    assert np.allclose(objs, ref["objective"], rtol=1e-14, atol=0.0)
    worst = int(np.argmin(np.where(np.arange(n) == ref["selected"][0], np.inf,
                                   [np.sum(v[nb[c]] * np.maximum(0.0, 3.0 - C[c, nb[c]])) for c in range(n)])))
    with pytest.raises(AssertionError):
        parity.replay_greedy_local(np.ascontiguousarray(C.T), v, 3.0, nb, [worst])

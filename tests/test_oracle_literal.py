"""The literal greedy step's oracle (Sec. 3.5, Eq. 11-15) against a
hand-derived toy, exact transport programs, a closed form and invariants."""
import json
import os

import numpy as np
import pytest

from oracle import literal, ot, sgs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "literal_toy.json")


def _toy():
    with open(GOLDEN) as f:
        return json.load(f)


@pytest.mark.parametrize("case", [0, 1])
def test_toy_matches_hand_derivation(case):
    g = _toy()
    C = np.array(g["cost_source_major"])
    v = np.array(g["tokens"]["capacity"])
    c = g["cases"][case]
    out = literal.literal_sgs_ref(C, v, c["K"], eps=0.01, rounds=4000)
    assert out["selected"].tolist() == c["selected"]
    assert np.allclose(out["score"], c["score"], atol=2e-6)
    assert np.allclose(out["residual"], c["residual"], atol=2e-6)
    if "objective" in c:
        assert out["objective"] == pytest.approx(c["objective"], abs=1e-4)


def test_toy_final_objective_matches_exact_transport():
    g = _toy()
    C = np.array(g["cost_source_major"])
    v = np.array(g["tokens"]["capacity"])
    out = literal.literal_sgs_ref(C, v, 3, eps=0.005, rounds=20000)
    S = out["selected"]
    exact, _ = ot.ot_lp(C[S], np.full(3, 1 / 3), v)
    assert out["objective"] == pytest.approx(exact, abs=0.01)
    assert out["objective"] >= exact - 1e-9


def _random(m, n, seed):
    rng = np.random.default_rng(seed)
    C = rng.uniform(0.0, 3.0, (m, n))
    v = rng.uniform(0.5, 1.5, n)
    return C, v / v.sum()


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_scaling_approaches_the_semi_relaxed_lp(seed):
    # As eps shrinks the entropic plan's cost approaches the exact semi-relaxed
    # optimum (Eq. 11) from above, within eps times log(mn).
    C, v = _random(3, 8, seed)
    u = np.full(3, 0.2)
    exact, _ = ot.sot_lp(C, u, v)
    for eps in (0.05, 0.01):
        a, b, E = literal.sot_scaling(C, u, v, eps, 20000)
        P = a[:, None] * E * b[None, :]
        assert np.allclose(P.sum(axis=1), u, rtol=1e-8)
        assert np.all(P.sum(axis=0) <= v * (1 + 1e-12))
        cost = float(np.sum(P * C))
        assert exact - 1e-9 <= cost <= exact + eps * np.log(C.size) + 1e-9


def test_single_source_is_water_filling():
    # One source of mass u: the optimum is P_j = min(v_j, lam exp(-C_j / eps))
    # with lam set by sum_j P_j = u (KKT of Eq. 12 with one row).
    rng = np.random.default_rng(5)
    n, eps, u = 12, 0.1, 0.3
    C = rng.uniform(0.0, 2.0, (1, n))
    v = rng.uniform(0.02, 0.15, n)
    w = np.exp(-C[0] / eps)
    lo, hi = 0.0, 1e6
    for _ in range(200):
        lam = 0.5 * (lo + hi)
        if np.minimum(v, lam * w).sum() > u:
            hi = lam
        else:
            lo = lam
    expect = np.minimum(v, lam * w)
    a, b, E = literal.sot_scaling(C, [u], v, eps, 500)
    P = (a[:, None] * E * b[None, :])[0]
    assert np.allclose(P, expect, rtol=1e-9, atol=1e-14)


def test_balanced_masses_give_the_entropic_ot_plan():
    # With sum u = sum v the capacity bound must be tight: both marginals hold
    # and log P + C / eps splits into a row part plus a column part.
    C, v = _random(4, 4, 7)
    u = np.full(4, 0.25)
    a, b, E = literal.sot_scaling(C, u, v, 0.2, 20000)
    P = a[:, None] * E * b[None, :]
    assert np.allclose(P.sum(axis=1), u, rtol=1e-9)
    assert np.allclose(P.sum(axis=0), v, rtol=1e-7)
    L = np.log(P) + C / 0.2
    resid = L - L.mean(axis=1, keepdims=True) - L.mean(axis=0, keepdims=True) + L.mean()
    assert np.abs(resid).max() < 1e-9


def test_first_pick_is_the_weighted_medoid():
    # Before any token is retained r = v, so the first pick minimises
    # sum_j v_j C(t, j), which is also the coverage-loss greedy's first pick.
    C, v = _random(30, 30, 9)
    np.fill_diagonal(C, 0.0)
    out = literal.literal_sgs_ref(C, v, 1, eps=0.05, rounds=10)
    assert out["selected"][0] == int(np.argmin(C @ v))
    assert out["selected"][0] == sgs.sgs_ref(C, v, 1, 3.0)["selected"][0]


def test_residual_mass_is_what_the_sources_leave():
    # At convergence the l retained tokens carry l/K, all of it within the
    # capacities, so the residual mass before pick l is 1 - l/K.
    C, v = _random(25, 25, 11)
    np.fill_diagonal(C, 0.0)
    K = 6
    out = literal.literal_sgs_ref(C, v, K, eps=0.1, rounds=3000)
    assert np.allclose(out["residual"], 1.0 - np.arange(K) / K, atol=1e-8)


def test_follow_replays_a_trajectory():
    C, v = _random(20, 20, 13)
    np.fill_diagonal(C, 0.0)
    own = literal.literal_sgs_ref(C, v, 5, eps=0.1, rounds=50)
    again = literal.literal_sgs_ref(C, v, 5, eps=0.1, rounds=50, follow=own["selected"])
    assert np.array_equal(again["selected"], own["selected"])
    assert np.array_equal(again["score"], own["best"])
    other = list(own["selected"][:4]) + [int(np.setdiff1d(np.arange(20), own["selected"])[0])]
    rep = literal.literal_sgs_ref(C, v, 5, eps=0.1, rounds=50, follow=other)
    assert rep["score"][4] >= rep["best"][4]
    with pytest.raises(ValueError):
        literal.literal_sgs_ref(C, v, 3, eps=0.1, rounds=5, follow=[1, 1, 2])


def test_steps_limit_is_a_prefix():
    C, v = _random(20, 20, 17)
    np.fill_diagonal(C, 0.0)
    full = literal.literal_sgs_ref(C, v, 6, eps=0.1, rounds=30)
    part = literal.literal_sgs_ref(C, v, 6, eps=0.1, rounds=30, steps=3)
    assert np.array_equal(part["selected"], full["selected"][:3])
    assert np.array_equal(part["score"], full["score"][:3])
    assert part["objective"] is None

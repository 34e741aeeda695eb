"""The capacity oracle (Sec. 3.4, Eq. 9-10) against a hand-derived toy,
library routines on special cases, and invariants."""
import json
import os

import numpy as np
import pytest
from scipy.spatial import cKDTree
from scipy.spatial.distance import cdist

from oracle import capacity
from scenes import make_scene, subscene

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "capacity_toy.json")


def _toy():
    with open(GOLDEN) as f:
        g = json.load(f)
    t = g["tokens"]
    return (np.array(t["features"]), np.array(t["positions"], np.float32), np.array(t["frames"], np.int32),
            g["cases"])


@pytest.mark.parametrize("case", [0, 1])
def test_toy_matches_hand_derivation(case):
    F, X, tau, cases = _toy()
    c = cases[case]
    out = capacity.capacity_ref(F, X, tau, c["n"])
    assert np.allclose(out["r"], c["r"], atol=1e-8)
    assert np.allclose(out["v"], c["v"], atol=1e-8)


def test_toy_temporal_orientation():
    # Swapping the orientation of d_tau changes the toy's scores: the
    # reading ReLU(tau_j - tau_k) is what the fixture pins.
    F, X, tau, cases = _toy()
    flipped = capacity.capacity_ref(F, X, -tau, 1)
    assert not np.allclose(flipped["r"], cases[0]["r"], atol=1e-3)


def _scene(n=400, seed=3):
    s = make_scene("n1024_d256_f32", seed)
    rng = np.random.default_rng(seed)
    return subscene(s, np.sort(rng.choice(s.n, n, replace=False)))


@pytest.mark.parametrize("n_nb", [1, 8, 16])
def test_spatial_term_is_mean_kdtree_distance(n_nb):
    # alpha = (0, 1, 0): r_j is proportional to the mean distance to the n
    # nearest other tokens, which a KD-tree gives directly.
    s = _scene()
    out = capacity.capacity_ref(s.feats, s.pos, s.frame, n_nb, alpha=(0, 1, 0))
    dist, _ = cKDTree(s.pos.astype(np.float64)).query(s.pos.astype(np.float64), k=n_nb + 1)
    mean = dist[:, 1:].mean(axis=1)
    assert np.allclose(out["v"], mean / mean.sum(), rtol=1e-12, atol=0)


@pytest.mark.parametrize("n_nb", [2, 16])
def test_feature_term_is_mean_cosine_distance(n_nb):
    # alpha = (1, 0, 0) on the KD-tree's neighbours: scipy's cosine distance.
    s = _scene(seed=4)
    dist, idx = cKDTree(s.pos.astype(np.float64)).query(s.pos.astype(np.float64), k=n_nb + 1)
    assert np.all(np.diff(dist, axis=1) > 0), "scene has distance ties; pick another seed"
    nb = idx[:, 1:]
    out = capacity.capacity_ref(s.feats, s.pos, s.frame, n_nb, alpha=(1, 0, 0))
    assert np.array_equal(out["neighbours"], nb)
    F = s.feats.astype(np.float64)
    d = np.array([cdist(F[j:j + 1], F[nb[j]], "cosine")[0] for j in range(s.n)])
    m = d.max()
    r = (d / m).mean(axis=1)
    assert np.allclose(out["r"], r, rtol=1e-12, atol=1e-15)
    assert out["maxima"][0] == pytest.approx(m, rel=1e-12)


def test_temporal_term_closed_form():
    # alpha = (0, 0, 1): r_j = mean over neighbours of ReLU(tau_j - tau_k) / M_tau.
    s = _scene(seed=5)
    out = capacity.capacity_ref(s.feats, s.pos, s.frame, 4, alpha=(0, 0, 1))
    nb = out["neighbours"]
    d = np.maximum(s.frame[:, None].astype(np.int64) - s.frame[nb], 0)
    r = d.mean(axis=1) / d.max()
    assert np.allclose(out["r"], r, rtol=1e-13, atol=0)


def test_invariants():
    s = _scene(seed=6)
    out = capacity.capacity_ref(s.feats, s.pos, s.frame, 8)
    v = out["v"]
    assert np.all(v >= 0) and v.sum() == pytest.approx(1.0, abs=1e-12)
    # Scaling space or rescaling features leaves every normalised term alone.
    scaled = capacity.capacity_ref(3.0 * s.feats, 2.0 * s.pos, s.frame, 8)
    assert np.array_equal(scaled["neighbours"], out["neighbours"])
    assert np.allclose(scaled["v"], v, rtol=1e-10)
    # Shifting every frame index by a constant changes nothing either.
    shifted = capacity.capacity_ref(s.feats, s.pos, s.frame + 7, 8)
    assert np.allclose(shifted["v"], v, rtol=1e-13)


def test_identical_tokens_give_uniform_capacity():
    F = np.ones((10, 4))
    X = np.zeros((10, 3), np.float32)
    tau = np.zeros(10, np.int32)
    out = capacity.capacity_ref(F, X, tau, 3)
    assert np.all(out["r"] == 0.0)
    assert np.allclose(out["v"], 0.1)


def test_self_is_never_a_neighbour():
    # A duplicated token's nearest other token is its twin at distance 0.
    s = _scene(n=50, seed=7)
    d = subscene(s, np.concatenate([np.arange(50), [10, 20]]))
    nb = capacity.neighbours_excluding_self(d.pos, 3)
    assert all(j not in nb[j] for j in range(d.n))
    assert nb[10][0] == 50 and nb[50][0] == 10 and nb[20][0] == 51


def test_distinct_tokens_weigh_more():
    # A token far from a tight cluster gets the largest capacity (Sec. 3.4:
    # locally distinctive tokens are prioritised).
    rng = np.random.default_rng(8)
    X = np.concatenate([rng.normal(0, 0.05, (30, 3)), [[5.0, 5.0, 5.0]]]).astype(np.float32)
    F = np.concatenate([np.tile([[1.0, 0.0]], (30, 1)) + rng.normal(0, 0.01, (30, 2)), [[0.0, 1.0]]])
    out = capacity.capacity_ref(F, X, np.zeros(31, np.int32), 4)
    assert int(np.argmax(out["v"])) == 30


def test_rejects_bad_n():
    F, X, tau, _ = _toy()
    with pytest.raises(ValueError):
        capacity.capacity_ref(F, X, tau, 4)
    with pytest.raises(ValueError):
        capacity.capacity_ref(F, X, tau, 0)

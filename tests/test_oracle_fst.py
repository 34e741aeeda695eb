"""Pins for the oracle's FST cost (Sec. 3.3, Eq. 7-8): hand-derived values,
library special cases, brute force and invariants."""
import math

import numpy as np
import pytest
from scipy.spatial.distance import cdist

from oracle import fst
from scenes import make_scene, subscene

# Toy scene (conftest ``toy``): f = (1,0), (1,0), (0,1), (1,1); x = (0,0,0),
# (1,0,0), (0,2,0), (2,2,0); tau = 0, 1, 1, 2; lam = 1, kappa = 10.
# By hand: M_f = 1 (tokens 0 and 2 are orthogonal), M_x = sqrt(8) (tokens 0
# and 3), M_tau = 2.  For example C(0, 1): d_f = 0, d_x = 1, d_tau = 0, so
# C = ln(1 + 10/sqrt(8)) / ln(11) = 0.630529; C(1, 0) adds ReLU(1 - 0)/2 = 0.5.
TOY_C = np.array([
    [0.000000, 0.630529, 1.870883, 1.292893],
    [1.130529, 0.000000, 1.911921, 1.204814],
    [2.370883, 1.911921, 0.000000, 1.163776],
    [2.292893, 1.704814, 1.663776, 0.000000],
])


def test_toy_hand_values(toy):
    C, (m_f, m_x, m_t) = fst.fst_cost_ref(toy["F"], toy["X"], toy["tau"])
    assert m_f == pytest.approx(1.0, abs=1e-15)
    assert m_x == pytest.approx(math.sqrt(8.0), rel=1e-15)
    assert m_t == 2.0
    assert np.allclose(C, TOY_C, atol=6e-7)
    assert C[0, 1] == pytest.approx(math.log(1 + 10 / math.sqrt(8)) / math.log(11), rel=1e-14)


def _scene(n=160, seed=3, cfg="n1024_d256_f32"):
    s = make_scene(cfg, seed)
    idx = np.random.default_rng(seed).choice(s.n, size=n, replace=False)
    return subscene(s, np.sort(idx))


def test_feature_term_is_scipy_cosine_distance():
    s = _scene()
    F = fst.widen_features(s.feats, s.dtype)
    C, (m_f, _, _) = fst.fst_cost_ref(F, s.pos, s.frame, weights=(1, 0, 0))
    ref = cdist(F, F, "cosine")
    np.fill_diagonal(ref, 0.0)
    assert m_f == pytest.approx(ref.max(), rel=1e-12)
    assert np.allclose(C, ref / ref.max(), atol=1e-12)


def test_spatial_term_is_scipy_euclidean_at_kappa_zero():
    s = _scene()
    F = fst.widen_features(s.feats, s.dtype)
    C, (_, m_x, _) = fst.fst_cost_ref(F, s.pos, s.frame, weights=(0, 1, 0), kappa=0.0)
    ref = cdist(s.pos.astype(np.float64), s.pos.astype(np.float64))
    assert m_x == pytest.approx(ref.max(), rel=1e-14)
    assert np.allclose(C, ref / ref.max(), atol=1e-14)


def test_phi_shape():
    z = np.linspace(0.0, 1.0, 101)
    for kappa in (0.5, 1.0, 10.0, 100.0):
        p = fst.phi(z, kappa)
        assert p[0] == 0.0 and p[-1] == pytest.approx(1.0, abs=1e-15)
        assert np.all(np.diff(p) > 0)                 # monotone increasing
        assert np.all(p[1:-1] > z[1:-1])              # concave: expands the near field
    assert np.allclose(fst.phi(z, 1e-9), z, atol=1e-9)  # kappa -> 0 limit is the identity


def test_temporal_term_brute_force():
    s = _scene(n=60)
    F = fst.widen_features(s.feats, s.dtype)
    C, (_, _, m_t) = fst.fst_cost_ref(F, s.pos, s.frame, weights=(0, 0, 1))
    tau = [int(t) for t in s.frame]
    span = max(tau) - min(tau)
    assert m_t == span
    for a in range(len(tau)):
        for b in range(len(tau)):
            assert C[a, b] == max(0, tau[a] - tau[b]) / span


@pytest.mark.parametrize("cfg", ["n1024_d256_f32", "n4096_d1152"])
def test_invariants(cfg):
    s = _scene(n=200, cfg=cfg)
    F = fst.widen_features(s.feats, s.dtype)
    lam = (1.0, 0.7, 0.4)
    C, (m_f, m_x, m_t) = fst.fst_cost_ref(F, s.pos, s.frame, weights=lam, kappa=10.0)
    assert np.all(np.diag(C) == 0.0)
    assert C.min() >= 0.0 and C.max() <= sum(lam) + 1e-12
    tau = s.frame.astype(np.float64)
    # Only the temporal term is asymmetric: C(i,j) - C(j,i) = lam_tau (tau_i - tau_j) / M_tau.
    assert np.allclose(C - C.T, lam[2] * (tau[:, None] - tau[None, :]) / m_t, atol=1e-12)
    # Each normalised term reaches exactly 1 on its maximising pair.
    for w in ((1, 0, 0), (0, 1, 0), (0, 0, 1)):
        Cw, _ = fst.fst_cost_ref(F, s.pos, s.frame, weights=w, kappa=10.0)
        assert Cw.max() == pytest.approx(1.0, abs=1e-15)


def test_zero_norm_feature_has_cosine_zero():
    s = _scene(n=40)
    F = fst.widen_features(s.feats, s.dtype)
    F[7] = 0.0
    d = fst.feature_discrepancy(F)
    assert d[7, 7] == 0.0
    assert np.all(np.delete(d[7], 7) == 1.0) and np.all(np.delete(d[:, 7], 7) == 1.0)


def test_rows_agree_with_full_matrix():
    s = _scene(n=300)
    F = fst.widen_features(s.feats, s.dtype)
    full, m = fst.fst_cost_ref(F, s.pos, s.frame)
    rows = np.array([0, 5, 17, 299])
    part, m2 = fst.fst_cost_ref(F, s.pos, s.frame, rows=rows)
    assert m == m2
    assert np.allclose(part, full[rows], rtol=0, atol=1e-14)   # BLAS may round a row subset differently
    assert np.array_equal(fst.target_major(full), full.T)


def test_bf16_widening_is_exact():
    bits = np.array([[0x3F80, 0xC000, 0x3F81, 0x0000, 0x7F7F]], np.uint16)
    got = fst.widen_features(bits, "bf16")[0]
    assert list(got[:4]) == [1.0, -2.0, 1.0078125, 0.0]
    assert got[4] == pytest.approx(3.3895313892515355e38, rel=1e-15)

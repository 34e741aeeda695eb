"""LP identities that tie the greedy's set function to the paper's transport
problems (Sec. 3.1 and 3.5, Eq. 2, 11)."""
import numpy as np
import pytest

from oracle import fst, ot, sgs
from scenes import make_scene, subscene


def _small(n, seed):
    s = make_scene("n1024_d256_f32", seed)
    s = subscene(s, np.sort(np.random.default_rng(seed).choice(s.n, n, replace=False)))
    F = fst.widen_features(s.feats, s.dtype)
    C, _ = fst.fst_cost_ref(F, s.pos, s.frame)
    return C, s.capacity.astype(np.float64)


@pytest.mark.parametrize("seed", range(4))
def test_semi_relaxed_equals_balanced_when_masses_match(seed):
    # With sum(u) = sum(v) the inequality P^T 1 <= v is tight (Sec. 3.5).
    rng = np.random.default_rng(seed)
    C = rng.random((4, 7))
    u = rng.random(4); u /= u.sum()
    v = rng.random(7); v /= v.sum()
    a, _ = ot.ot_lp(C, u, v)
    b, _ = ot.sot_lp(C, u, v)
    assert a == pytest.approx(b, rel=1e-9)


@pytest.mark.parametrize("seed", range(4))
def test_coverage_loss_is_free_source_transport(seed):
    # The greedy's L(S) is the transport cost with the retained tokens' masses
    # free: each target's capacity goes whole to its cheapest retained token.
    C, v = _small(12, seed)
    rng = np.random.default_rng(seed)
    S = sorted(rng.choice(12, size=4, replace=False).tolist())
    lp, P = ot.free_source_lp(C[S], v)
    assert sgs.coverage_loss(C, v, S, 3.0) == pytest.approx(lp, rel=1e-9)


def test_relaxed_loss_bounds_balanced_loss():
    # Freeing the source masses can only lower the cost: L(S) <= L_OT(S).
    C, v = _small(10, 9)
    for S in ([0, 3], [1, 2, 5], [4, 6, 7, 9]):
        u = np.full(len(S), 1.0 / len(S))
        bal, _ = ot.ot_lp(C[S], u, v)
        assert sgs.coverage_loss(C, v, S, 3.0) <= bal + 1e-9

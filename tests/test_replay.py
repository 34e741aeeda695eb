"""The guided replay that checks GPU greedy trajectories at full size
(tests/parity.py): on small inputs it must agree with evaluating every
candidate at every step, accept exactly the valid trajectories and reject a
planted wrong pick (CPU only)."""
import numpy as np
import pytest

from oracle import sgs
from tests import parity


def _random_case(n, seed):
    rng = np.random.default_rng(seed)
    C = rng.random((n, n)) * 3.0
    np.fill_diagonal(C, 0.0)
    v = rng.random(n)
    return C, v / v.sum()


@pytest.mark.parametrize("n,k,seed", [(50, 10, 0), (200, 60, 1), (300, 300, 2), (64, 1, 3)])
def test_lazy_replay_of_the_oracle_greedy(n, k, seed):
    C, v = _random_case(n, seed)
    ref = sgs.sgs_ref(C, v, k, 3.0)
    ties, g, o, near = parity.lazy_replay(C, v, 3.0, ref["selected"])
    assert ties == [] and near == []
    assert np.array_equal(g, ref["gain"]) and np.array_equal(o, ref["objective"])
    t2, g2, o2 = parity.replay_greedy(C, v, 3.0, ref["selected"])
    assert t2 == [] and np.array_equal(g, g2) and np.array_equal(o, o2)


def test_lazy_replay_rejects_a_wrong_pick():
    C, v = _random_case(120, 4)
    sel = sgs.sgs_ref(C, v, 30, 3.0)["selected"].copy()
    # Swap step 5's pick for the 10th pick: a strictly worse gain at step 5.
    sel[5], sel[9] = sel[9], sel[5]
    with pytest.raises(AssertionError, match="step 5"):
        parity.lazy_replay(C, v, 3.0, sel)
    with pytest.raises(AssertionError, match="step 5"):
        parity.replay_greedy(C, v, 3.0, sel)


def test_lazy_replay_rejects_repeats_and_bad_indices():
    C, v = _random_case(40, 5)
    with pytest.raises(AssertionError):
        parity.lazy_replay(C, v, 3.0, [3, 3])
    with pytest.raises(AssertionError):
        parity.lazy_replay(C, v, 3.0, [40])


def test_lazy_replay_lists_exact_ties():
    # Token 60 is a twin of token 7 (same costs both ways) and token 7 covers
    # everything cheaply, so both have the best gain at step 0: picking the
    # twin with the larger index is a valid greedy step, listed as a tie.
    C, v = _random_case(61, 6)
    C[7] *= 0.1
    C[60] = C[7]
    C[:, 60] = C[:, 7]
    C[7, 60] = C[60, 7] = C[60, 60] = 0.0
    assert int(sgs.sgs_ref(C, v, 1, 3.0)["selected"][0]) == 7
    ties, g, o, near = parity.lazy_replay(C, v, 3.0, [60])
    assert ties == [0] and near[0]["oracle"] == 7 and near[0]["gain"] == near[0]["oracle_gain"]
    t2, g2, _ = parity.replay_greedy(C, v, 3.0, [60])
    assert t2 == [0] and np.array_equal(g, g2)


def test_lazy_replay_with_an_alternative_cost():
    # Picks made greedily on a perturbed cost are accepted against the true
    # cost once the propagated error is allowed, and rejected without it when
    # the perturbation changes a pick.
    C, v = _random_case(150, 7)
    rng = np.random.default_rng(8)
    for _ in range(20):
        A = np.clip(C + rng.uniform(-2e-3, 2e-3, C.shape), 0.0, None)
        np.fill_diagonal(A, 0.0)
        picks = sgs.sgs_ref(A, v, 40, 3.0)["selected"]
        ties, g, o, near = parity.lazy_replay(C, v, 3.0, picks, alt=A)
        # The replay's gains are the true cost's, along the perturbed picks.
        t2, g2, o2 = parity.replay_greedy(C, v, 3.0, picks, tie_atol=np.inf)
        assert np.array_equal(g, g2) and np.array_equal(o, o2) and ties == t2
        if ties:
            with pytest.raises(AssertionError):
                parity.lazy_replay(C, v, 3.0, picks, tie_rtol=0.0)
            break
    else:
        pytest.fail("no perturbation changed a pick")


def test_oracle_cost_full_is_the_oracle():
    from scenes import make_scene, subscene
    s = make_scene("n4096_d1152", 3)
    s = subscene(s, np.arange(0, 4096, 5))
    C, m = parity.oracle_cost_full(s, block=100)
    C2, m2 = parity.oracle_cost(s)
    assert np.array_equal(C, C2) and m == m2


def test_threaded_neighbour_table_is_the_oracle():
    from oracle import capacity
    from scenes import make_scene
    s = make_scene("n1024_d256_f32", 2)
    a = parity.oracle_neighbours_excluding_self(s.pos, 8, block=100)
    b = capacity.neighbours_excluding_self(s.pos, 8)
    assert np.array_equal(a, b)

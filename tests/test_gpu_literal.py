"""GPU parity of coverprune_sgs_literal_select against the literal-step
oracle (Sec. 3.5, Eq. 11-15)."""
import json
import os

import numpy as np
import pytest

from scenes import make_scene
from oracle import literal
from tests import parity

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "literal_toy.json")

# Both sides work in float64 and differ only in the order of additions; a
# pick may differ from the oracle's only between scores this close.
SCORE_RTOL = 1e-9


def _cp():
    import paper_2608_13226_amd as cp
    return cp


def _gpu(C_src, v, k, eps, rounds, follow=None, steps=True):
    cost = torch.from_numpy(np.ascontiguousarray(np.asarray(C_src, np.float32).T)).cuda()
    cap = torch.from_numpy(np.ascontiguousarray(v, dtype=np.float32)).cuda()
    f = None if follow is None else torch.from_numpy(np.asarray(follow, np.int32)).cuda()
    r = _cp().sgs_literal_select(cost, cap, k, epsilon=eps, rounds=rounds, follow=f, steps=steps)
    torch.cuda.synchronize()
    return (r.selected.cpu().numpy(), r.score.cpu().numpy(), r.residual.cpu().numpy(),
            float(r.objective.cpu().numpy()[0]))


def _eps(eps):
    """The float32 value the library receives, for the oracle."""
    return float(np.float32(eps))


def _compare(C32, v, k, eps, rounds):
    """GPU trajectory replayed by the oracle: every pick within SCORE_RTOL of
    the oracle's best, scores and residuals alike, the same objective; and the
    oracle's own trajectory when no pick needed the tolerance."""
    C = C32.astype(np.float64)
    sel, score, resid, obj = _gpu(C32, v, k, eps, rounds)
    rep = literal.literal_sgs_ref(C, v.astype(np.float64), k, _eps(eps), rounds, follow=sel)
    assert len(set(sel.tolist())) == k
    assert np.all(rep["score"] <= rep["best"] + SCORE_RTOL * np.abs(rep["best"]) + 1e-15)
    assert np.allclose(score, rep["score"], rtol=SCORE_RTOL, atol=1e-12)
    assert np.allclose(resid, rep["residual"], rtol=1e-9, atol=1e-12)
    assert obj == pytest.approx(rep["objective"], rel=1e-9)
    ties = np.nonzero(rep["score"] != rep["best"])[0]
    if len(ties) == 0:
        own = literal.literal_sgs_ref(C, v.astype(np.float64), k, _eps(eps), rounds)
        assert np.array_equal(sel, own["selected"])
    return sel, ties


@pytest.mark.parametrize("case", [0, 1])
def test_literal_toy(case):
    with open(GOLDEN) as f:
        g = json.load(f)
    C = np.array(g["cost_source_major"], np.float32)
    v = np.array(g["tokens"]["capacity"], np.float32)
    c = g["cases"][case]
    print(f"literal toy K={c['K']}", flush=True)
    sel, score, resid, obj = _gpu(C, v, c["K"], 0.01, 4000)
    assert sel.tolist() == c["selected"]
    assert np.allclose(score, c["score"], atol=2e-6)
    assert np.allclose(resid, c["residual"], atol=2e-6)
    if "objective" in c:
        assert obj == pytest.approx(c["objective"], abs=1e-4)


# (config, tokens, k, eps, rounds, seed)
CASES = [
    ("n1024_d256_f32", 300, 30, 0.05, 50, 0),
    ("n4096_d1152", 997, 60, 0.05, 20, 1),       # ragged: 64-row blocks and 256-column strips
    ("n4096_d1152", 500, 40, 0.2, 100, 2),
    ("n8192_d3584", 1200, 25, 0.02, 200, 3),
]


@pytest.mark.parametrize("cfg,n,k,eps,rounds,seed", CASES)
def test_literal_matches_oracle(cfg, n, k, eps, rounds, seed):
    s = parity.sample_scene(cfg, n, seed, salt=5000)
    print(f"literal {cfg} n={s.n} k={k} eps={eps} rounds={rounds}", flush=True)
    C_ref, _ = parity.oracle_cost(s)
    _, ties = _compare(C_ref.astype(np.float32), s.capacity, k, eps, rounds)
    assert len(ties) <= 1


def test_literal_edge_cases():
    s = parity.sample_scene("n1024_d256_f32", 64, 4, salt=5000)
    C32 = parity.oracle_cost(s)[0].astype(np.float32)
    v = s.capacity
    print("literal k = 1, k = n, one round", flush=True)
    sel, score, resid, _ = _gpu(C32, v, 1, 0.05, 10)
    w = C32.astype(np.float64) @ v.astype(np.float64)
    assert sel[0] == int(np.argmin(w)) and score[0] == pytest.approx(w.min(), rel=1e-12)
    assert resid[0] == pytest.approx(float(v.astype(np.float64).sum()), rel=1e-12)
    _compare(C32, v, 64, 0.1, 5)          # every token retained
    _compare(C32, v, 12, 0.1, 1)          # a single scaling round per solve


def test_literal_follow_prices_a_given_set():
    s = parity.sample_scene("n4096_d1152", 400, 6, salt=5000)
    C32 = parity.oracle_cost(s)[0].astype(np.float32)
    v = s.capacity
    rng = np.random.default_rng(6)
    given = rng.choice(s.n, 30, replace=False)
    print("literal follow", flush=True)
    sel, _, _, obj = _gpu(C32, v, 30, 0.05, 60, follow=given, steps=False)
    assert np.array_equal(sel, given)
    ref = literal.literal_sgs_ref(C32.astype(np.float64), v.astype(np.float64), 30, _eps(0.05), 60, follow=given)
    assert obj == pytest.approx(ref["objective"], rel=1e-9)
    sel2, score2, _, obj2 = _gpu(C32, v, 30, 0.05, 60, follow=given, steps=True)
    assert np.array_equal(sel2, given) and obj2 == pytest.approx(obj, rel=1e-12)
    assert np.allclose(score2, ref["score"], rtol=SCORE_RTOL)


def test_literal_deterministic():
    s = parity.sample_scene("n4096_d1152", 700, 7, salt=5000)
    C32 = parity.oracle_cost(s)[0].astype(np.float32)
    print("literal determinism", flush=True)
    a = _gpu(C32, s.capacity, 40, 0.05, 30)
    b = _gpu(C32, s.capacity, 40, 0.05, 30)
    for x, y in zip(a[:3], b[:3]):
        assert np.array_equal(x, y)
    assert a[3] == b[3]


@pytest.mark.slow
def test_literal_full_size_first_steps():
    # 16384 tokens, K = 1638: the whole run on the GPU, its first 4 steps
    # replayed by the oracle on the same float32 cost (narrow features keep
    # the oracle's cost fast).
    s = make_scene("n16384_d3584", 0, dim=16)
    print(f"literal full size n={s.n} k={s.k}", flush=True)
    C_tm, _ = parity.oracle_cost_f32_target_major(s)
    cost = torch.from_numpy(C_tm).cuda()
    cap = torch.from_numpy(s.capacity).cuda()
    r = _cp().sgs_literal_select(cost, cap, s.k, epsilon=0.05, rounds=20)
    torch.cuda.synchronize()
    sel = r.selected.cpu().numpy()
    assert len(set(sel.tolist())) == s.k
    assert np.isfinite(r.objective.cpu().numpy()[0])
    rep = literal.literal_sgs_ref(C_tm.T.astype(np.float64), s.capacity.astype(np.float64), s.k, _eps(0.05), 20,
                                  follow=sel, steps=4)
    assert np.all(rep["score"] <= rep["best"] + SCORE_RTOL * rep["best"])
    assert np.allclose(r.score.cpu().numpy()[:4], rep["score"], rtol=SCORE_RTOL)
    assert np.allclose(r.residual.cpu().numpy()[:4], rep["residual"], rtol=1e-9)

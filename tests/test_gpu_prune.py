"""coverprune_prune (Sec. 3: the FST cost of Eq. 7-8, then the greedy of Sec.
3.5) against the two calls it stands for, and against the oracle.

For n a multiple of 64 the cost's epilogue also writes the greedy's
source-major copy of the cost and its step-0 gains (fixed-point partial sums
over blocks of 64 targets); the greedy then starts without a first pass of its
own.  The result must be bit for bit that of coverprune_fst_cost followed by
coverprune_sgs_select(CP_SGS_INCREMENTAL): the same cost, picks, gains,
objective and assignment.  Other sizes run the two calls' kernels in turn.
"""
import numpy as np
import pytest

from oracle import sgs
from scenes import make_scene, to_device
from tests import parity

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _cp():
    import paper_2608_13226_amd as cp
    return cp


def _both(t, cap, k, c0=None):
    cp = _cp()
    cost, mx, r = cp.prune(t["feats"], t["pos"], t["frame"], cap, k, c0=c0)
    cost2, mx2 = cp.fst_cost(t["feats"], t["pos"], t["frame"])
    r2 = cp.sgs_select(cost2, cap, k, c0=c0, incremental=True)
    torch.cuda.synchronize()
    assert torch.equal(cost, cost2)
    assert torch.equal(mx, mx2)
    for a, b in zip((r.selected, r.gain, r.objective, r.assign), (r2.selected, r2.gain, r2.objective, r2.assign)):
        assert torch.equal(a, b)
    return cost, r


# (config, tokens, k, seed): multiples of 64 (the fused epilogue), one of them
# an odd number of 64-token tiles, and a ragged size (the two calls' kernels).
CASES = [
    ("n4096_d1152", 1024, 100, 0),
    ("n4096_d1152", 1536, 200, 1),
    ("n4096_d1152", 1000, 100, 2),
    ("n8192_d3584", 2048, 300, 3),        # past the candidate lists' start
]


@pytest.mark.parametrize("cfg,n,k,seed", CASES)
def test_prune_matches_two_calls(cfg, n, k, seed):
    s = parity.sample_scene(cfg, n, seed, salt=3000)
    print(f"prune vs two calls cfg={cfg} n={s.n} k={k} seed={seed}", flush=True)
    t = to_device(s)
    _both(t, t["capacity"], k)


def test_prune_skewed_capacity():
    # One token holds most of the capacity: the fixed-point scale is then set
    # by the largest single term rather than by the total.
    s = parity.sample_scene("n4096_d1152", 1024, 5, salt=3000)
    v = np.full(s.n, 1e-4, np.float32)
    v[17] = 1.0
    v /= v.sum()
    print(f"prune skewed capacity n={s.n}", flush=True)
    t = to_device(s)
    _both(t, torch.from_numpy(v).cuda(), 64)


def test_prune_end_to_end_oracle():
    # The fused path against the oracle's own float64 cost and greedy: a pick
    # may differ only where two gains lie closer than the cost error resolves.
    s = parity.sample_scene("n4096_d1152", 1024, 7, salt=3000)
    k = 120
    print(f"prune end to end n={s.n} k={k}", flush=True)
    t = to_device(s)
    cost, _, r = _cp().prune(t["feats"], t["pos"], t["frame"], t["capacity"], k, c0=3.0)
    torch.cuda.synchronize()
    sel = r.selected.cpu().numpy()
    C_ref, _ = parity.oracle_cost(s)
    err = np.abs(cost.cpu().numpy().T.astype(np.float64) - C_ref).max()
    ties, _, o_or = parity.replay_greedy(C_ref, s.capacity, 3.0, sel, tie_atol=2 * err)
    ref = sgs.sgs_ref(C_ref, s.capacity.astype(np.float64), k, 3.0)
    assert abs(o_or[-1] - ref["objective"][-1]) <= 1e-3 * ref["objective"][-1]
    assert np.allclose(r.objective.cpu().numpy(), o_or, rtol=1e-4)
    print(f"  {len(ties)} near-tie steps", flush=True)


@pytest.mark.slow
def test_prune_full_workload():
    # The benchmark's scene and launch shape (16384 tokens, K = 1638).
    s = make_scene("n16384_d3584", 0)
    print(f"prune full workload n={s.n} k={s.k}", flush=True)
    t = to_device(s)
    _both(t, t["capacity"], s.k)

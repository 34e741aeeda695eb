"""GPU parity of coverprune_sgs_select against the oracle greedy (Eq. 11-16)."""
import numpy as np
import pytest

from scenes import make_scene, subscene, to_device
from oracle import sgs
from tests import parity

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _cp():
    import paper_2608_13226_amd as cp
    return cp


def _sub(cfg, n, seed):
    return parity.sample_scene(cfg, n, seed, salt=2000)


# Both forms of the greedy: full sweeps (dense) and running gains updated from
# the targets whose best cost drops (incremental), the latter in both
# schedules: every block finds the improved targets from the pick's row of
# the transposed cost ("rows"), or the blocks exchange them ("compact").
MODES = ["dense", "rows", "compact"]


def _run(cost, cap, k, c0, mode):
    return _cp().sgs_select(cost, cap, k, c0=c0, incremental=mode != "dense", compact=mode == "compact")


def _gpu_select(C_tm_f32: np.ndarray, v: np.ndarray, k: int, c0: float, mode="dense"):
    cost = torch.from_numpy(np.ascontiguousarray(C_tm_f32)).cuda()
    cap = torch.from_numpy(np.ascontiguousarray(v, dtype=np.float32)).cuda()
    r = _run(cost, cap, k, c0, mode)
    torch.cuda.synchronize()
    return (r.selected.cpu().numpy(), r.gain.cpu().numpy(), r.objective.cpu().numpy(),
            r.assign.cpu().numpy())


def _same_cost_case(s, k, c0=3.0, weights=(1.0, 1.0, 1.0), kappa=10.0, mode="dense"):
    """The oracle's cost, rounded once to float32, drives both greedies."""
    C_ref, _ = parity.oracle_cost(s, weights, kappa)
    C32 = C_ref.astype(np.float32)                 # source-major, float32 values
    v = s.capacity
    ref = sgs.sgs_ref(C32.astype(np.float64), v.astype(np.float64), k, c0)
    sel, gain, obj, assign = _gpu_select(np.ascontiguousarray(C32.T), v, k, c0, mode)
    ties, g_or, o_or = parity.replay_greedy(C32, v, c0, sel)
    assert np.allclose(gain, g_or, rtol=1e-6, atol=1e-12)
    assert np.allclose(obj, o_or, rtol=1e-9, atol=1e-12)
    if not ties:
        assert np.array_equal(sel, ref["selected"])
        assert np.array_equal(assign, ref["assign"])
    parity.check_trajectory_invariants(sel, gain, obj, v, c0, k, s.n)
    return ties


# (config, tokens, k, seed): ragged tails for the 256-column strips and the row
# chunks, odd sizes (scalar path), float32 and bfloat16 derived costs.
CASES = [
    ("n1024_d256_f32", None, 102, 0),
    ("n1024_d256_f32", None, 102, 1),
    ("n4096_d1152", 1000, 100, 0),
    ("n4096_d1152", 997, 150, 1),
    ("n8192_d3584", 1531, 60, 2),
    ("n16384_d3584", 300, 300, 3),         # k = n
    ("n16384_d3584", 64, 1, 4),            # k = 1
]


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("cfg,n,k,seed", CASES)
def test_same_cost_parity(cfg, n, k, seed, mode):
    s = _sub(cfg, n, seed)
    print(f"sgs same-cost {cfg} n={s.n} k={k} seed={seed} mode={mode}", flush=True)
    ties = _same_cost_case(s, k, mode=mode)
    assert len(ties) <= 1, f"unexpected near-ties at steps {ties}"


@pytest.mark.parametrize("mode", MODES)
def test_single_token(mode):
    s = _sub("n4096_d1152", 1, 0)
    s.capacity[:] = 1.0
    print(f"sgs n=1 mode={mode}", flush=True)
    sel, gain, obj, assign = _gpu_select(np.zeros((1, 1), np.float32), s.capacity, 1, 3.0, mode)
    assert sel.tolist() == [0] and assign.tolist() == [0]
    assert gain[0] == pytest.approx(3.0) and obj[0] == 0.0


@pytest.mark.parametrize("mode", MODES)
def test_exact_ties_go_to_smaller_index(mode):
    # Duplicated tokens have identical gains at every step; the smaller index wins.
    s = _sub("n4096_d1152", 200, 5)
    idx = np.concatenate([np.arange(200), np.arange(0, 200, 7)])
    d = subscene(s, idx)
    print(f"sgs exact ties mode={mode}", flush=True)
    C_ref, _ = parity.oracle_cost(d)
    C32 = C_ref.astype(np.float32)
    ref = sgs.sgs_ref(C32.astype(np.float64), d.capacity.astype(np.float64), 40, 3.0)
    sel, _, _, _ = _gpu_select(np.ascontiguousarray(C32.T), d.capacity, 40, 3.0, mode)
    assert np.array_equal(sel, ref["selected"])


@pytest.mark.parametrize("mode", MODES)
def test_zero_capacity_steps_still_select(mode):
    # Only 3 targets carry capacity: after they are covered every gain is 0 and
    # the remaining picks go to the smallest unselected indices.
    s = _sub("n4096_d1152", 120, 6)
    v = np.zeros(120, np.float32)
    v[[5, 50, 99]] = np.float32(1 / 3)
    s.capacity = v
    print("sgs zero-gain steps", flush=True)
    C_ref, _ = parity.oracle_cost(s)
    C32 = C_ref.astype(np.float32)
    ref = sgs.sgs_ref(C32.astype(np.float64), v.astype(np.float64), 10, 3.0)
    sel, gain, _, _ = _gpu_select(np.ascontiguousarray(C32.T), v, 10, 3.0, mode)
    assert np.array_equal(sel, ref["selected"])
    assert np.all(gain[3:] == 0.0)


@pytest.mark.parametrize("mode", MODES)
def test_end_to_end_parity(mode):
    # GPU cost and GPU greedy against the oracle's cost and greedy.  A pick may
    # differ from the oracle's only where two gains are closer than the cost
    # error can resolve.
    s = _sub("n4096_d1152", 1200, 7)
    k = 120
    print(f"sgs end-to-end n={s.n} k={k} mode={mode}", flush=True)
    t = to_device(s)
    cp = _cp()
    cost, _ = cp.fst_cost(t["feats"], t["pos"], t["frame"])
    r = _run(cost, t["capacity"], k, 3.0, mode)
    torch.cuda.synchronize()
    sel = r.selected.cpu().numpy()
    C_ref, _ = parity.oracle_cost(s)
    err = np.abs(cost.cpu().numpy().T.astype(np.float64) - C_ref).max()
    ties, _, o_or = parity.replay_greedy(C_ref, s.capacity, 3.0, sel, tie_atol=2 * err)
    ref = sgs.sgs_ref(C_ref, s.capacity.astype(np.float64), k, 3.0)
    assert abs(o_or[-1] - ref["objective"][-1]) <= 1e-3 * ref["objective"][-1]
    assert np.allclose(r.objective.cpu().numpy(), o_or, rtol=1e-4)
    print(f"  {len(ties)} near-tie steps", flush=True)


@pytest.mark.parametrize("mode", MODES)
def test_lists_that_do_not_fit(mode):
    # Past step 128 the rows schedule continues from candidate lists when
    # they fit.  Here they cannot: a candidate's cost to every other target
    # falls with its index, so once the greedy has picked candidate m, every
    # candidate above m undercuts the best cost of nearly all targets (about
    # five candidates keep 300 to 700 such pairs after 128 picks, above the
    # 255 a list holds).  The rows of T then serve the remaining steps (the
    # gated second launch), with the same result.
    n, k = 1024, 200
    rng = np.random.default_rng(21)
    C_src = np.repeat((1.0 - 1e-3 * np.arange(n) / n)[:, None], n, axis=1)
    C_src = (C_src + 1e-5 * rng.random((n, n))).astype(np.float32)
    np.fill_diagonal(C_src, 0.0)
    v = rng.random(n).astype(np.float32)
    v /= v.sum()
    print(f"sgs lists that do not fit, mode={mode}", flush=True)
    ref = sgs.sgs_ref(C_src.astype(np.float64), v.astype(np.float64), k, 3.0)
    sel, gain, obj, assign = _gpu_select(np.ascontiguousarray(C_src.T), v, k, 3.0, mode)
    ties, g_or, o_or = parity.replay_greedy(C_src, v, 3.0, sel)
    assert np.allclose(gain, g_or, rtol=1e-6, atol=1e-12)
    assert np.allclose(obj, o_or, rtol=1e-9, atol=1e-12)
    if not ties:
        assert np.array_equal(sel, ref["selected"]) and np.array_equal(assign, ref["assign"])


@pytest.mark.parametrize("mode", MODES)
def test_deterministic(mode):
    s = _sub("n4096_d1152", 1000, 8)
    C_ref, _ = parity.oracle_cost(s)
    C_tm = np.ascontiguousarray(C_ref.T.astype(np.float32))
    print(f"sgs determinism mode={mode}", flush=True)
    a = _gpu_select(C_tm, s.capacity, 100, 3.0, mode)
    b = _gpu_select(C_tm, s.capacity, 100, 3.0, mode)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


@pytest.mark.slow
@pytest.mark.parametrize("mode", MODES)
def test_full_size_first_steps(mode):
    # 16384 tokens, the benchmark's launch shape, first 6 steps against the
    # oracle on the same float32 cost (narrow 16-d features keep the oracle fast).
    s = make_scene("n16384_d3584", 0, dim=16)
    print(f"sgs full size n={s.n} mode={mode}", flush=True)
    C_tm, _ = parity.oracle_cost_f32_target_major(s)
    k = 6
    sel, gain, obj, _ = _gpu_select(C_tm, s.capacity, k, 3.0, mode)
    C32 = C_tm.T
    ties, g_or, o_or = parity.replay_greedy(C32, s.capacity, 3.0, sel)
    assert np.allclose(gain, g_or, rtol=1e-6)
    assert np.allclose(obj, o_or, rtol=1e-9)
    assert not ties


@pytest.mark.slow
def test_incremental_general_form_matches_oracle():
    # Beyond the benchmark's size: a seeded random cost of 16900 tokens (W = 67
    # rows and columns per block, two column groups per block in the rows
    # schedule), every form replayed against the oracle.
    n, k = 16900, 24
    print(f"sgs incremental general form n={n} k={k}", flush=True)
    rng = np.random.default_rng(11)
    C_src = rng.random((n, n), dtype=np.float32) * np.float32(3.0)
    np.fill_diagonal(C_src, 0.0)
    v = np.full(n, 1.0 / n, np.float32)
    cost = torch.from_numpy(C_src).cuda().t().contiguous()
    cap = torch.from_numpy(v).cuda()
    out = {mode: _run(cost, cap, k, 3.0, mode) for mode in MODES}
    torch.cuda.synchronize()
    res = {m: (r.selected.cpu().numpy(), r.gain.cpu().numpy(), r.objective.cpu().numpy(), r.assign.cpu().numpy())
           for m, r in out.items()}
    del cost, out
    for mode, (sel, gain, obj, assign) in res.items():
        ties, g_or, o_or, near = parity.lazy_replay(C_src, v, 3.0, sel)
        print(f"  {mode}: near-ties {near}", flush=True)
        assert np.allclose(gain, g_or, rtol=1e-6, atol=1e-12)
        assert np.allclose(obj, o_or, rtol=1e-9, atol=1e-12)
        parity.check_trajectory_invariants(sel, gain, obj, v, 3.0, k, n)
    for x, y in zip(res["rows"], res["compact"]):
        assert np.array_equal(x, y)

"""GPU parity of coverprune_sgs_select_batch: several scenes' greedies in one
launch give each scene the picks of its own incremental greedy and of the
oracle (Sec. 3.5, Eq. 11-16)."""
import numpy as np
import pytest

from scenes import make_scene, to_device
from oracle import sgs
from tests import parity

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _cp():
    import paper_2608_13226_amd as cp
    return cp


def _case(cfg, n, seed):
    s = parity.sample_scene(cfg, n, seed, salt=6000)
    C32 = parity.oracle_cost(s)[0].astype(np.float32)      # source-major float32 values
    return s, C32


# Both schedules of the incremental form: improved targets found by every
# block from the transposed cost ("rows") or exchanged between blocks.
SCHEDULES = [pytest.param(False, id="rows"), pytest.param(True, id="compact")]


def _run_batch(cases, ks, c0=3.0, compact=False):
    costs = [torch.from_numpy(np.ascontiguousarray(C.T)).cuda() for _, C in cases]
    caps = [torch.from_numpy(np.ascontiguousarray(s.capacity)).cuda() for s, _ in cases]
    res = _cp().sgs_select_batch(costs, caps, ks, c0=c0, compact=compact)
    single = [_cp().sgs_select(c, v, k, c0=c0, incremental=True, compact=compact)
              for c, v, k in zip(costs, caps, ks)]
    torch.cuda.synchronize()
    return res, single


def _np(r):
    return r.selected.cpu().numpy(), r.gain.cpu().numpy(), r.objective.cpu().numpy(), r.assign.cpu().numpy()


def _check_scene(s, C32, k, got, alone, c0=3.0):
    sel, gain, obj, assign = _np(got)
    a_sel, a_gain, a_obj, a_assign = _np(alone)
    # The scene alone and in the batch: the same exact fixed-point greedy.
    assert np.array_equal(sel, a_sel)
    assert np.array_equal(gain, a_gain) and np.array_equal(obj, a_obj)
    assert np.array_equal(assign, a_assign)
    # Against the oracle, as for the single-scene greedy.
    ties, g_or, o_or = parity.replay_greedy(C32, s.capacity, c0, sel)
    assert np.allclose(gain, g_or, rtol=1e-6, atol=1e-12)
    assert np.allclose(obj, o_or, rtol=1e-9, atol=1e-12)
    if not ties:
        ref = sgs.sgs_ref(C32.astype(np.float64), s.capacity.astype(np.float64), k, c0)
        assert np.array_equal(sel, ref["selected"])
        assert np.array_equal(assign, ref["assign"])


@pytest.mark.parametrize("compact", SCHEDULES)
def test_batch_of_mixed_sizes(compact):
    specs = [("n1024_d256_f32", 300, 30, 0), ("n4096_d1152", 997, 100, 1), ("n8192_d3584", 1531, 60, 2),
             ("n4096_d1152", 64, 64, 3)]
    cases = [_case(cfg, n, seed) for cfg, n, _, seed in specs]
    ks = [k for _, _, k, _ in specs]
    print(f"sgs batch sizes {[s.n for s, _ in cases]} ks {ks} compact={compact}", flush=True)
    res, single = _run_batch(cases, ks, compact=compact)
    for (s, C32), k, got, alone in zip(cases, ks, res, single):
        _check_scene(s, C32, k, got, alone)


def test_batch_of_one():
    cases = [_case("n4096_d1152", 1000, 4)]
    print("sgs batch of one", flush=True)
    res, single = _run_batch(cases, [100])
    _check_scene(*cases[0], 100, res[0], single[0])


@pytest.mark.parametrize("compact", SCHEDULES)
def test_batch_of_sixteen(compact):
    # The largest batch: sixteen small scenes, including n = 1, k = 1 and k = n.
    rng = np.random.default_rng(5)
    sizes = [1, 2, 40, 64, 65, 100, 128, 129, 200, 257, 300, 333, 64, 90, 150, 400]
    cases = [_case("n4096_d1152", n, 10 + i) for i, n in enumerate(sizes)]
    ks = [max(1, min(n, int(rng.integers(1, n + 1)))) for n in sizes]
    ks[3], ks[4] = 64, 1
    print(f"sgs batch of sixteen ks {ks} compact={compact}", flush=True)
    res, single = _run_batch(cases, ks, compact=compact)
    for (s, C32), k, got, alone in zip(cases, ks, res, single):
        _check_scene(s, C32, k, got, alone)


def test_batch_deterministic():
    cases = [_case("n4096_d1152", 800, 20), _case("n1024_d256_f32", 500, 21)]
    print("sgs batch determinism", flush=True)
    a, _ = _run_batch(cases, [80, 50])
    b, _ = _run_batch(cases, [80, 50])
    for x, y in zip(a, b):
        for u, w in zip(_np(x), _np(y)):
            assert np.array_equal(u, w)


@pytest.mark.slow
def test_batch_paper_shape():
    # Four scenes of the paper's 6272-token (32 x 196) shape, K = 628, costs
    # from the GPU's own FST kernel: each scene's picks in the batch equal its
    # picks alone, and each trajectory is replayed against the oracle's own
    # float64 cost, with the cost error propagated into the tie allowance.
    cp = _cp()
    scenes = [make_scene("paper_n6272_d3584", seed) for seed in range(4)]
    costs, caps = [], []
    for s in scenes:
        t = to_device(s)
        c, _ = cp.fst_cost(t["feats"], t["pos"], t["frame"])
        costs.append(c)
        caps.append(t["capacity"])
    ks = [s.k for s in scenes]
    print(f"sgs batch paper shape n={scenes[0].n} k={ks[0]} x {len(scenes)}", flush=True)
    res = cp.sgs_select_batch(costs, caps, ks)
    single = [cp.sgs_select(c, v, k, incremental=True) for c, v, k in zip(costs, caps, ks)]
    torch.cuda.synchronize()
    for s, got, alone, cost in zip(scenes, res, single, costs):
        sel, gain, obj = got.selected.cpu().numpy(), got.gain.cpu().numpy(), got.objective.cpu().numpy()
        assert np.array_equal(sel, alone.selected.cpu().numpy())
        assert np.array_equal(gain, alone.gain.cpu().numpy())
        parity.check_trajectory_invariants(sel, gain, obj, s.capacity, 3.0, s.k, s.n)
        C_ref, _ = parity.oracle_cost_full(s)
        C_gpu = cost.t().contiguous().cpu().numpy()
        ties, g_or, o_or, near = parity.lazy_replay(C_ref, s.capacity, 3.0, sel, alt=C_gpu)
        print(f"  seed {s.seed}: near-ties {[(x['step'], x['pick'], x['oracle']) for x in near]}", flush=True)
        assert np.allclose(obj, o_or, rtol=1e-4, atol=1e-9)

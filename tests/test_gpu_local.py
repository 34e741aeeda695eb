"""GPU parity of coverprune_knn and coverprune_sgs_local_select against the
oracle (Sec. 3.5, Eq. 13): neighbour tables bit for bit, local-greedy picks
against the oracle greedy restricted to the same tables."""
import numpy as np
import pytest

from scenes import make_scene, subscene
from oracle import knn as oknn
from oracle import sgs
from tests import parity

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _cp():
    import paper_2608_13226_amd as cp
    return cp


def _sub(cfg, n, seed):
    return parity.sample_scene(cfg, n, seed, salt=3000)


def _gpu_knn(pos: np.ndarray, g: int) -> np.ndarray:
    p = torch.from_numpy(np.ascontiguousarray(pos, dtype=np.float32)).cuda()
    out = _cp().knn(p, g)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def _gpu_local(C_tm_f32: np.ndarray, v: np.ndarray, nbr: np.ndarray, k: int, c0: float):
    cost = torch.from_numpy(np.ascontiguousarray(C_tm_f32, dtype=np.float32)).cuda()
    cap = torch.from_numpy(np.ascontiguousarray(v, dtype=np.float32)).cuda()
    nb = torch.from_numpy(np.ascontiguousarray(nbr, dtype=np.int32)).cuda()
    r = _cp().sgs_local_select(cost, cap, nb, k, c0=c0)
    torch.cuda.synchronize()
    return (r.selected.cpu().numpy(), r.gain.cpu().numpy(), r.objective.cpu().numpy(),
            r.assign.cpu().numpy())


# ---------------------------------------------------------------------------
# Neighbour tables.

KNN_CASES = [
    ("n1024_d256_f32", None, 1, 0),        # g = 1: every token's own index
    ("n1024_d256_f32", None, 16, 1),
    ("n4096_d1152", 997, 64, 2),           # ragged: not a multiple of the block
    ("n4096_d1152", 1000, 128, 6),         # largest g of the bounding pass
    ("n4096_d1152", 1000, 129, 7),         # smallest g of the radix select
    ("n4096_d1152", 300, 300, 3),          # g = n: the whole scene, sorted
    ("n8192_d3584", 2048, 1024, 4),        # largest g
    ("n16384_d3584", 1, 1, 5),             # one token
]


@pytest.mark.parametrize("cfg,n,g,seed", KNN_CASES)
def test_knn_matches_oracle(cfg, n, g, seed):
    s = _sub(cfg, n, seed)
    print(f"knn {cfg} n={s.n} g={g} seed={seed}", flush=True)
    got = _gpu_knn(s.pos, g)
    ref = oknn.knn_ref(s.pos, g)
    assert np.array_equal(got, ref)


def test_knn_exact_ties_on_a_grid():
    # Integer lattice: many exactly equal distances, broken by index.
    ax = np.arange(7, dtype=np.float32)
    pos = np.stack(np.meshgrid(ax, ax, ax, indexing="ij"), -1).reshape(-1, 3)
    rng = np.random.default_rng(12)
    pos = pos[rng.permutation(len(pos))]
    print(f"knn lattice n={len(pos)}", flush=True)
    for g in (1, 7, 27, 100):
        assert np.array_equal(_gpu_knn(pos, g), oknn.knn_ref(pos, g))


def test_knn_duplicate_positions():
    # Repeated tokens sit at distance 0 from each other; the smaller index first.
    s = _sub("n4096_d1152", 200, 13)
    idx = np.concatenate([np.arange(200), np.arange(0, 200, 3), np.arange(0, 200, 9)])
    d = subscene(s, idx)
    print(f"knn duplicates n={d.n}", flush=True)
    assert np.array_equal(_gpu_knn(d.pos, 40), oknn.knn_ref(d.pos, 40))


def test_knn_coincident_tokens_take_the_radix_path():
    # Every token at one point: all distances are 0, every row is 0..g-1, and
    # the bounding pass collects all n tokens per row, more than it keeps, so
    # every row is redone by the radix select.
    pos = np.full((600, 3), 1.25, np.float32)
    print("knn coincident tokens", flush=True)
    got = _gpu_knn(pos, 24)
    assert np.array_equal(got, np.tile(np.arange(24), (600, 1)))
    assert np.array_equal(got, oknn.knn_ref(pos, 24))


def test_knn_half_coincident():
    # Half the tokens share one point (rows there overflow the bounding pass),
    # the rest are spread out (rows there do not).
    s = _sub("n4096_d1152", 800, 20)
    pos = s.pos.copy()
    pos[::2] = pos[0]
    print("knn half coincident", flush=True)
    for g in (8, 64, 200):
        assert np.array_equal(_gpu_knn(pos, g), oknn.knn_ref(pos, g))


def test_knn_full_size_sampled_rows():
    # The 16384-token scene at the local greedy's g = 64 and at the largest g,
    # sampled rows against the oracle.
    s = make_scene("n16384_d3584", 0, dim=16)
    rng = np.random.default_rng(14)
    rows = np.sort(rng.choice(s.n, 256, replace=False))
    for g in (64, 128, 1024):
        print(f"knn full size n={s.n} g={g}", flush=True)
        got = _gpu_knn(s.pos, g)
        assert np.array_equal(got[rows], oknn.knn_ref(s.pos, g, rows=rows))


@pytest.mark.slow
def test_knn_beyond_keys_in_lds():
    # 32768 tokens, more than the radix select keeps in LDS: its rows recompute
    # their keys from the positions.  A quarter of the tokens share one point,
    # so their rows overflow the bounding pass and take the radix select; g =
    # 200 sends every row there.  Sampled rows against the oracle.
    s = make_scene("lite_n32768_d3584", 0, dim=8)
    pos = s.pos.copy()
    pos[::4] = pos[0]
    rng = np.random.default_rng(15)
    rows = np.sort(np.concatenate([rng.choice(s.n, 96, replace=False), np.arange(0, 128, 4)]))
    for g in (17, 200):
        print(f"knn n={s.n} g={g} (keys recomputed)", flush=True)
        got = _gpu_knn(pos, g)
        assert np.array_equal(got[rows], oknn.knn_ref(pos, g, rows=rows))


# ---------------------------------------------------------------------------
# Local greedy on the oracle's cost and the oracle's neighbour tables.

def _local_case(s, k, g, c0=3.0, nbr=None):
    C_ref, _ = parity.oracle_cost(s)
    C32 = C_ref.astype(np.float32)                 # source-major, float32 values
    v = s.capacity
    if nbr is None:
        nbr = oknn.knn_ref(s.pos, g)
    ref = sgs.sgs_ref(C32.astype(np.float64), v.astype(np.float64), k, c0, neighbours=nbr)
    C_tm = np.ascontiguousarray(C32.T)
    sel, gain, obj, assign = _gpu_local(C_tm, v, nbr, k, c0)
    ties, g_or, o_or = parity.replay_greedy_local(C_tm, v, c0, nbr, sel)
    # Terms are float64 products summed in exact fixed point: gains and L agree
    # with the oracle's float64 sums to rounding.
    assert np.allclose(gain, g_or, rtol=1e-12, atol=1e-15)
    assert np.allclose(obj, o_or, rtol=1e-12, atol=1e-15)
    assert not ties, f"near-ties at steps {ties}"
    assert np.array_equal(sel, ref["selected"])
    assert np.allclose(gain, ref["gain"], rtol=1e-12, atol=1e-15)
    assert np.array_equal(assign, ref["assign"])
    # The objective falls by at least the local gain at every step.
    total = c0 * float(np.sum(v, dtype=np.float64))
    prev = np.concatenate([[total], obj[:-1]])
    assert np.all(prev - obj >= gain - 1e-12 * total)
    return sel


# (config, tokens, k, g, seed)
LOCAL_CASES = [
    ("n1024_d256_f32", None, 102, 16, 0),
    ("n4096_d1152", 1000, 100, 64, 1),
    ("n4096_d1152", 997, 150, 128, 2),     # largest g, ragged
    ("n8192_d3584", 1531, 60, 1, 3),       # g = 1: a token's gain is its own term
    ("n16384_d3584", 300, 300, 32, 4),     # k = n
    ("n16384_d3584", 64, 1, 64, 5),        # g = n, k = 1
]


@pytest.mark.parametrize("cfg,n,k,g,seed", LOCAL_CASES)
def test_local_same_cost_parity(cfg, n, k, g, seed):
    s = _sub(cfg, n, seed)
    print(f"sgs local {cfg} n={s.n} k={k} g={g} seed={seed}", flush=True)
    _local_case(s, k, g)


def test_local_with_all_targets_is_the_dense_greedy():
    # g = n: every target is a neighbour, so the local form is the dense one.
    s = _sub("n4096_d1152", 128, 15)
    C_ref, _ = parity.oracle_cost(s)
    C_tm = np.ascontiguousarray(C_ref.astype(np.float32).T)
    nbr = oknn.knn_ref(s.pos, s.n)
    print("sgs local g = n against the dense greedy", flush=True)
    a = _gpu_local(C_tm, s.capacity, nbr, 40, 3.0)
    cost = torch.from_numpy(C_tm).cuda()
    cap = torch.from_numpy(s.capacity).cuda()
    r = _cp().sgs_select(cost, cap, 40, c0=3.0)
    torch.cuda.synchronize()
    assert np.array_equal(a[0], r.selected.cpu().numpy())
    assert np.allclose(a[1], r.gain.cpu().numpy(), rtol=1e-6)
    assert np.array_equal(a[3], r.assign.cpu().numpy())


def test_local_arbitrary_table():
    # Any table of distinct targets, not only nearest neighbours.
    s = _sub("n4096_d1152", 500, 16)
    rng = np.random.default_rng(16)
    nbr = np.stack([rng.choice(s.n, 24, replace=False) for _ in range(s.n)])
    print("sgs local arbitrary table", flush=True)
    _local_case(s, 60, 24, nbr=nbr)


def test_local_exact_ties_go_to_smaller_index():
    s = _sub("n4096_d1152", 200, 17)
    idx = np.concatenate([np.arange(200), np.arange(0, 200, 7)])
    d = subscene(s, idx)
    print("sgs local exact ties", flush=True)
    _local_case(d, 40, 32)


def test_local_zero_capacity_steps_still_select():
    s = _sub("n4096_d1152", 120, 18)
    v = np.zeros(120, np.float32)
    v[[5, 50, 99]] = np.float32(1 / 3)
    s.capacity = v
    print("sgs local zero-gain steps", flush=True)
    sel = _local_case(s, 10, 16)
    assert len(set(sel.tolist())) == 10


def test_local_single_token():
    v = np.ones(1, np.float32)
    sel, gain, obj, assign = _gpu_local(np.zeros((1, 1), np.float32), v, np.zeros((1, 1), np.int32), 1, 3.0)
    assert sel.tolist() == [0] and assign.tolist() == [0]
    assert gain[0] == pytest.approx(3.0) and obj[0] == 0.0


def test_local_deterministic():
    s = _sub("n4096_d1152", 1000, 19)
    C_ref, _ = parity.oracle_cost(s)
    C_tm = np.ascontiguousarray(C_ref.T.astype(np.float32))
    nbr = oknn.knn_ref(s.pos, 64)
    print("sgs local determinism", flush=True)
    a = _gpu_local(C_tm, s.capacity, nbr, 100, 3.0)
    b = _gpu_local(C_tm, s.capacity, nbr, 100, 3.0)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


@pytest.mark.slow
def test_local_full_size():
    # 16384 tokens, g = 64, the full K = 1638 steps, on the oracle's float32
    # cost (narrow 16-d features keep the oracle fast) and the oracle's tables.
    s = make_scene("n16384_d3584", 0, dim=16)
    g = 64
    print(f"sgs local full size n={s.n} k={s.k} g={g}", flush=True)
    C_tm, _ = parity.oracle_cost_f32_target_major(s)
    nbr = np.concatenate([oknn.knn_ref(s.pos, g, rows=np.arange(a, min(s.n, a + 1024)))
                          for a in range(0, s.n, 1024)])
    sel, gain, obj, assign = _gpu_local(C_tm, s.capacity, nbr, s.k, 3.0)
    # The replay asserts that every pick is the best local gain or within
    # 1e-6 (relative) of it; over 1638 steps the kernel's 64-bit fixed-point
    # sums (resolution 2^-62 c0 sum v) may order a near-tie differently from
    # float64 sums, after which both follow the kernel's own trajectory.
    ties, g_or, o_or = parity.replay_greedy_local(C_tm, s.capacity, 3.0, nbr, sel)
    print(f"  {len(ties)} near-tie steps", flush=True)
    assert np.allclose(gain, g_or, rtol=1e-12, atol=1e-15)
    assert np.allclose(obj, o_or, rtol=1e-12, atol=1e-15)
    assert len(set(sel.tolist())) == s.k

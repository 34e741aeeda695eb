"""GPU parity of coverprune_lite_select against the oracle (Eq. 17-20)."""
import numpy as np
import pytest

from scenes import make_scene, subscene, to_device
from tests import parity

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _cp():
    import paper_2608_13226_amd as cp
    return cp


def _sub(cfg, n, seed):
    return parity.sample_scene(cfg, n, seed, salt=3000)


def _gpu(s, k, h, weights=(1.0, 1.0, 1.0), kappa=10.0):
    t = to_device(s)
    r = _cp().lite_select(t["feats"], t["pos"], t["frame"], t["capacity"], k, weights=weights,
                          kappa=kappa, voxel_size=h, token_cost=True, check=True)
    return (r.selected.cpu().numpy(), r.group.cpu().numpy(), float(r.objective.cpu().numpy()[0]),
            r.token_cost.cpu().numpy())


CASES = [
    # (config, tokens, k, voxel, seed)
    ("n4096_d1152", 1000, 100, 0.25, 0),
    ("n4096_d1152", 1000, 100, 0.5, 1),
    ("n4096_d1152", 997, 37, 0.25, 2),
    ("n1024_d256_f32", None, 102, 0.25, 0),
    ("lite_n32768_d3584", 3000, 300, 0.25, 0),
    ("n16384_d3584", 2500, 250, 0.25, 1),      # capacity proportional to object size
    ("n8192_d3584", 800, 1, 0.25, 3),          # one group
    ("n8192_d3584", 300, 300, 0.25, 4),        # one token per group
    ("n8192_d3584", 500, 50, 100.0, 5),        # every token in one voxel
]


@pytest.mark.parametrize("cfg,n,k,h,seed", CASES)
def test_lite_matches_oracle(cfg, n, k, h, seed):
    s = _sub(cfg, n, seed)
    print(f"lite parity {cfg} n={s.n} k={k} h={h} seed={seed}", flush=True)
    ref = parity.lite_reference(s, k, h=h)
    sel, group, obj, tc = _gpu(s, k, h)
    ties = parity.assert_lite_close(sel, group, obj, ref, tc)
    print(f"  {ties} groups with another prototype of equal cost within the measured error", flush=True)


@pytest.mark.parametrize("weights,kappa", [((1.0, 0.0, 0.0), 10.0), ((0.0, 1.0, 1.0), 0.0),
                                           ((0.5, 2.0, 1.0), 3.0)])
def test_lite_weights(weights, kappa):
    s = _sub("n4096_d1152", 900, 6)
    print(f"lite weights={weights} kappa={kappa}", flush=True)
    ref = parity.lite_reference(s, 90, weights=weights, kappa=kappa, h=0.25)
    sel, group, obj, tc = _gpu(s, 90, 0.25, weights, kappa)
    parity.assert_lite_close(sel, group, obj, ref, tc)


def test_lite_skewed_capacity():
    # A few heavy tokens make groups of very different sizes (some above 16, the
    # MFMA tile height), and some thresholds are crossed twice in one token.
    s = _sub("n4096_d1152", 1500, 7)
    rng = np.random.default_rng(7)
    v = rng.random(s.n) ** 8
    s.capacity = (v / v.sum()).astype(np.float32)
    print("lite skewed capacity", flush=True)
    ref = parity.lite_reference(s, 60, h=0.25)
    sizes = np.bincount(ref["group"])
    assert sizes.max() > 16
    sel, group, obj, tc = _gpu(s, 60, 0.25)
    parity.assert_lite_close(sel, group, obj, ref, tc)


@pytest.mark.parametrize("cluster", [3000, 5000])
def test_lite_dense_cluster(cluster):
    # Most of 5200 tokens packed around one point: with 3000 there, one block's
    # span of whole buckets holds about 3100 tokens (the largest span the
    # front sorts in LDS, 16 per thread); with 5000 no span fits and the
    # stable radix sort orders the keys instead.
    s = _sub("n8192_d3584", 5200, 9)
    rng = np.random.default_rng(9)
    idx = rng.choice(s.n, size=cluster, replace=False)
    s.pos[idx] = (s.pos.mean(0) + rng.normal(scale=1e-4, size=(cluster, 3))).astype(np.float32)
    print(f"lite dense cluster of {cluster} in n={s.n}", flush=True)
    ref = parity.lite_reference(s, 520, h=0.25)
    sel, group, obj, tc = _gpu(s, 520, 0.25)
    parity.assert_lite_close(sel, group, obj, ref, tc)


def test_lite_keys_wider_than_the_bucket_pass():
    # A voxel of 1e-6 m puts every coordinate at the 21-bit clamp range: keys
    # of 63 bits do not pack with a token index into 64 bits, so the radix
    # sort runs; clamped keys tie and stay in token order.
    s = _sub("n4096_d1152", 1000, 10)
    print("lite tiny voxel", flush=True)
    ref = parity.lite_reference(s, 100, h=1e-6)
    sel, group, obj, tc = _gpu(s, 100, 1e-6)
    parity.assert_lite_close(sel, group, obj, ref, tc)


@pytest.mark.parametrize("n,k", [(1, 1), (2, 1), (2, 2), (3, 2), (17, 5), (257, 30)])
def test_lite_tiny_scenes(n, k):
    # One front block (two at 257 tokens), a token field of 0-9 bits, spans of
    # a single bucket and groups of one token.
    s = _sub("n4096_d1152", n, 11)
    print(f"lite tiny n={n} k={k}", flush=True)
    ref = parity.lite_reference(s, k, h=0.25)
    sel, group, obj, tc = _gpu(s, k, 0.25)
    parity.assert_lite_close(sel, group, obj, ref, tc)


def test_lite_identical_positions():
    # Every key is zero (a zero-width bucket field: one bucket holds every
    # token, sorted by index alone) and M_x is zero.
    s = _sub("n4096_d1152", 600, 12)
    s.pos[:] = s.pos[0]
    print("lite identical positions", flush=True)
    ref = parity.lite_reference(s, 60, h=0.25)
    sel, group, obj, tc = _gpu(s, 60, 0.25)
    parity.assert_lite_close(sel, group, obj, ref, tc)


def test_lite_deterministic():
    s = _sub("n4096_d1152", 1000, 8)
    print("lite determinism", flush=True)
    a = _gpu(s, 100, 0.25)
    b = _gpu(s, 100, 0.25)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1]) and a[2] == b[2]
    assert np.array_equal(a[3], b[3])


@pytest.mark.slow
@pytest.mark.parametrize("capacity", ["uniform", "fst16"])
def test_lite_full_size(capacity):
    # The full 32768-token Lite workload in the benchmark's launch shape, with
    # the generator's uniform capacities (groups of 9 and 10 tokens) and with
    # the workload's own FST capacities (16 neighbours, from the oracle),
    # whose groups range from 2 to 26 tokens.
    s = parity.workload_scene("lite_n32768_d3584", 0) if capacity == "fst16" else make_scene("lite_n32768_d3584", 0)
    print(f"lite full size n={s.n} k={s.k} capacity={capacity}", flush=True)
    if capacity == "fst16":
        # The library's own capacity at this size against the oracle's (the
        # input used below): within one float32 rounding.
        t = to_device(s)
        v_gpu, _ = _cp().fst_capacity(t["feats"], t["pos"], t["frame"], 16)
        v_gpu = v_gpu.cpu().numpy().astype(np.float64)
        assert np.allclose(v_gpu, s.capacity.astype(np.float64), rtol=2.0 ** -22, atol=0.0)
    sel, group, obj, tc = _gpu(s, s.k, 0.25)
    ref = parity.lite_reference(s, s.k, h=0.25)
    sizes = np.bincount(ref["group"])
    print(f"  group sizes {sizes.min()}..{sizes.max()}", flush=True)
    ties = parity.assert_lite_close(sel, group, obj, ref, tc)
    print(f"  {ties} groups with another prototype of equal cost within the measured error", flush=True)

"""GPU parity of coverprune_fst_capacity against the capacity oracle
(Sec. 3.4, Eq. 9-10)."""
import json
import os

import numpy as np
import pytest

from scenes import make_scene, subscene, to_device
from oracle import capacity, fst
from tests import parity

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "capacity_toy.json")


def _cp():
    import paper_2608_13226_amd as cp
    return cp


def _gpu(feats_t, pos, frame, n_nb, alpha=(1.0, 1.0, 1.0)):
    p = torch.from_numpy(np.ascontiguousarray(pos, dtype=np.float32)).cuda()
    f = torch.from_numpy(np.ascontiguousarray(frame, dtype=np.int32)).cuda()
    v, r = _cp().fst_capacity(feats_t, p, f, n_nb, alpha=alpha)
    torch.cuda.synchronize()
    return v.cpu().numpy(), r.cpu().numpy()


def _feats_t(scene):
    return to_device(scene)["feats"]


def _check(v, r, ref):
    # Scores: float64 sums of float64 terms; only the order of additions differs.
    assert np.allclose(r, ref["r"], rtol=1e-12, atol=1e-15)
    # Capacity: the float64 quotient rounded once to float32.
    assert np.allclose(v, ref["v"], rtol=2 ** -23, atol=0.0)
    assert abs(float(np.sum(v, dtype=np.float64)) - 1.0) <= 1e-6


def _scene_case(cfg, n, seed, n_nb, alpha=(1.0, 1.0, 1.0)):
    s = parity.sample_scene(cfg, n, seed, salt=4000)
    F = fst.widen_features(s.feats, s.dtype)
    ref = capacity.capacity_ref(F, s.pos, s.frame, n_nb, alpha=alpha)
    v, r = _gpu(_feats_t(s), s.pos, s.frame, n_nb, alpha)
    _check(v, r, ref)


CASES = [
    ("n1024_d256_f32", None, 0, 8),        # float32 features
    ("n1024_d256_f32", 300, 1, 1),
    ("n4096_d1152", 997, 2, 16),           # bf16, ragged
    ("n8192_d3584", 2048, 3, 16),          # bf16 at the LLM width
    ("n4096_d1152", 200, 4, 199),          # every other token is a neighbour
    ("n4096_d1152", 600, 5, 150),          # tables through the radix select
]


@pytest.mark.parametrize("cfg,n,seed,n_nb", CASES)
def test_capacity_matches_oracle(cfg, n, seed, n_nb):
    print(f"capacity {cfg} n={n} seed={seed} n_nb={n_nb}", flush=True)
    _scene_case(cfg, n, seed, n_nb)


@pytest.mark.parametrize("alpha", [(0.0, 1.0, 0.0), (1.0, 0.0, 0.0), (0.0, 0.0, 1.0), (2.0, 0.5, 1.5)])
def test_capacity_weights(alpha):
    print(f"capacity alpha={alpha}", flush=True)
    _scene_case("n4096_d1152", 800, 6, 8, alpha)


@pytest.mark.parametrize("case", [0, 1])
def test_capacity_toy(case):
    # The hand-derived four-token scene, features padded with zeros to d = 4.
    with open(GOLDEN) as f:
        g = json.load(f)
    t = g["tokens"]
    F = np.zeros((4, 4), np.float32)
    F[:, :2] = np.array(t["features"], np.float32)
    c = g["cases"][case]
    print(f"capacity toy n={c['n']}", flush=True)
    v, r = _gpu(torch.from_numpy(F).cuda(), np.array(t["positions"], np.float32), np.array(t["frames"]), c["n"])
    assert np.allclose(r, c["r"], atol=1e-8)
    assert np.allclose(v, c["v"], atol=1e-7)


def test_capacity_duplicates_and_zero_rows():
    # Twins (a token's nearest other is its copy at distance 0) and zero
    # feature rows (cos = 0, d_f = 1).
    s = parity.sample_scene("n1024_d256_f32", 300, 7, salt=4000)
    d = subscene(s, np.concatenate([np.arange(300), np.arange(0, 300, 5)]))
    feats = d.feats.copy()
    feats[[3, 17, 301]] = 0.0
    d.feats = feats
    print("capacity duplicates and zero rows", flush=True)
    ref = capacity.capacity_ref(fst.widen_features(d.feats, d.dtype), d.pos, d.frame, 6)
    v, r = _gpu(_feats_t(d), d.pos, d.frame, 6)
    _check(v, r, ref)


def test_capacity_identical_tokens_are_uniform():
    # Width 4: |f| = 2 exactly, so every discrepancy is exactly 0 and v falls
    # back to uniform.
    n = 50
    F = torch.ones((n, 4), dtype=torch.float32, device="cuda")
    v, r = _gpu(F, np.zeros((n, 3), np.float32), np.zeros(n, np.int32), 4)
    assert np.all(r == 0.0)
    assert np.all(v == np.float32(1.0 / n))


def test_capacity_identical_tokens_rounding():
    # Width 8: sqrt(8)^2 rounds above 8, so 1 - cos is a rounding residue that
    # the normalisation turns into 1 for every pair, in the oracle and here.
    n = 50
    F = np.ones((n, 8), np.float32)
    pos, tau = np.zeros((n, 3), np.float32), np.zeros(n, np.int32)
    ref = capacity.capacity_ref(F.astype(np.float64), pos, tau, 4)
    v, r = _gpu(torch.from_numpy(F).cuda(), pos, tau, 4)
    _check(v, r, ref)


def test_capacity_two_tokens():
    F = torch.tensor([[1.0, 0.0, 0.0, 0.0], [0.0, 1.0, 0.0, 0.0]], device="cuda")
    v, r = _gpu(F, np.array([[0, 0, 0], [1, 0, 0]], np.float32), np.array([0, 1]), 1)
    # pairs (0,1): d_f 1, d_x 1, d_tau 0; (1,0): 1, 1, 1 -> r = [2, 3], v = [0.4, 0.6]
    assert np.allclose(r, [2.0, 3.0], rtol=1e-15)
    assert np.allclose(v, [0.4, 0.6], rtol=1e-7)


def test_capacity_deterministic():
    s = parity.sample_scene("n4096_d1152", 2000, 8, salt=4000)
    f = _feats_t(s)
    print("capacity determinism", flush=True)
    a = _gpu(f, s.pos, s.frame, 16)
    b = _gpu(f, s.pos, s.frame, 16)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


@pytest.mark.slow
def test_capacity_full_size():
    # The 16384-token, 3584-d bf16 scene with 16 neighbours per token.
    s = make_scene("n16384_d3584", 0)
    print(f"capacity full size n={s.n} d={s.dim}", flush=True)
    v, r = _gpu(_feats_t(s), s.pos, s.frame, 16)
    F = fst.widen_features(s.feats, s.dtype)
    ref = capacity.capacity_ref(F, s.pos, s.frame, 16)
    _check(v, r, ref)

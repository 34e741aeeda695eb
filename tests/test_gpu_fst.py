"""GPU parity of coverprune_fst_cost against the float64 oracle (Eq. 7-8)."""
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
    return parity.sample_scene(cfg, n, seed, salt=1000)


def _run(scene, weights=(1.0, 1.0, 1.0), kappa=10.0):
    t = to_device(scene)
    cost, maxima = _cp().fst_cost(t["feats"], t["pos"], t["frame"], weights=weights, kappa=kappa)
    torch.cuda.synchronize()
    return cost.cpu().numpy(), maxima.cpu().numpy()


# (config, tokens or None for the whole scene, seed): several 128-tiles plus a
# ragged tail, an odd count, and float32 and bfloat16 features; from 4096
# tokens up, bf16 problems take the 256 x 256 tile path (whole tiles, and a
# ragged tail).
CASES = [
    ("n1024_d256_f32", None, 0),
    ("n1024_d256_f32", None, 1),
    ("n1024_d256_f32", 333, 2),
    ("n4096_d1152", 1000, 0),
    ("n4096_d1152", 997, 1),
    ("n8192_d3584", 700, 0),
    ("n16384_d3584", 520, 3),
    ("n4096_d1152", None, 0),
    ("n8192_d3584", 4357, 1),
]


@pytest.mark.parametrize("cfg,n,seed", CASES)
def test_cost_matches_oracle(cfg, n, seed):
    s = _sub(cfg, n, seed)
    print(f"fst_cost parity {cfg} n={s.n} seed={seed}", flush=True)
    C_ref, m_ref = parity.oracle_cost(s)
    C_gpu, m_gpu = _run(s)
    parity.assert_cost_close(C_gpu, C_ref)
    assert m_gpu[0] == pytest.approx(m_ref[0], rel=1e-5)
    assert m_gpu[1] == pytest.approx(m_ref[1], rel=1e-6)
    assert m_gpu[2] == m_ref[2]
    assert np.all(np.diag(C_gpu) == 0.0)


@pytest.mark.parametrize("weights,kappa", [((1.0, 0.0, 0.0), 10.0), ((0.0, 1.0, 0.0), 0.0),
                                           ((0.0, 0.0, 1.0), 10.0), ((0.7, 1.3, 0.4), 100.0),
                                           ((2.0, 0.5, 1.0), 1.0)])
def test_cost_weights_and_kappa(weights, kappa):
    s = _sub("n4096_d1152", 600, 4)
    print(f"fst_cost weights={weights} kappa={kappa}", flush=True)
    C_ref, _ = parity.oracle_cost(s, weights, kappa)
    C_gpu, _ = _run(s, weights, kappa)
    parity.assert_cost_close(C_gpu, C_ref)


def test_single_and_pair_tokens():
    s = _sub("n4096_d1152", 2, 0)
    for n in (1, 2):
        sub = subscene(s, np.arange(n))
        print(f"fst_cost n={n}", flush=True)
        C_ref, m_ref = parity.oracle_cost(sub)
        C_gpu, m_gpu = _run(sub)
        parity.assert_cost_close(C_gpu, C_ref)
        assert np.allclose(m_gpu, m_ref, rtol=1e-5)


def test_degenerate_scene():
    # One shared position and frame: M_x = M_tau = 0 zero their terms; a zero
    # feature row has cosine 0 with everything.
    s = _sub("n1024_d256_f32", 150, 5)
    s.pos[:] = s.pos[0]
    s.frame[:] = 3
    s.feats[17] = 0.0
    print("fst_cost degenerate scene", flush=True)
    C_ref, m_ref = parity.oracle_cost(s)
    C_gpu, m_gpu = _run(s)
    assert m_ref[1] == 0.0 and m_ref[2] == 0.0
    parity.assert_cost_close(C_gpu, C_ref)
    assert m_gpu[1] == 0.0 and m_gpu[2] == 0.0


def test_deterministic():
    s = _sub("n4096_d1152", 1000, 6)
    print("fst_cost determinism", flush=True)
    a, _ = _run(s)
    b, _ = _run(s)
    assert np.array_equal(a, b)


@pytest.mark.slow
def test_full_size_sampled_rows():
    # Full 16384-token scene in the benchmark's launch shape: oracle maxima over
    # all pairs, oracle costs from a sample of sources to every target.  Each
    # source row crosses the diagonal, so both triangles (written by different
    # code paths) are covered.
    s = make_scene("n16384_d3584", 0)
    print(f"fst_cost full size n={s.n}", flush=True)
    t = to_device(s)
    cost, maxima = _cp().fst_cost(t["feats"], t["pos"], t["frame"])
    rows = np.array([0, 1, 777, 8191, 12345, s.n - 1])
    gpu = cost[:, torch.from_numpy(rows).cuda()].cpu().numpy()     # [t, s in rows] = C(s, t)
    m_gpu = maxima.cpu().numpy()
    del cost
    from oracle import fst
    F = fst.widen_features(s.feats, s.dtype)
    m_ref = fst.sample_maxima(F, s.pos, s.frame, block=1024)
    assert m_gpu[0] == pytest.approx(m_ref[0], rel=1e-5)
    assert m_gpu[1] == pytest.approx(m_ref[1], rel=1e-6)
    assert m_gpu[2] == m_ref[2]
    C_rows, _ = fst.fst_cost_ref(F, s.pos, s.frame, rows=rows, maxima=m_ref)
    parity.assert_cost_close(gpu, C_rows)

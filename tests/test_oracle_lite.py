"""Pins for the oracle's CoverPrune-Lite (Sec. 4, Eq. 17-20): Morton code
values, closed-form group sizes, an independent scan formulation of the
grouping, hand-derived toy values, reduction to the full cost, and the block
transport LP of Eq. 19-20."""
import math

import numpy as np
import pytest

from oracle import fst, lite, ot
from scenes import make_scene, subscene


def test_morton_values():
    # Standard 3D Z-order interleave with x in the lowest bit.
    assert lite.morton_key(1, 0, 0) == 1
    assert lite.morton_key(0, 1, 0) == 2
    assert lite.morton_key(0, 0, 1) == 4
    assert lite.morton_key(1, 1, 1) == 7
    assert lite.morton_key(2, 0, 0) == 8
    assert lite.morton_key(3, 5, 7) == 431
    top = 2 ** 21 - 1
    assert lite.morton_key(top, top, top) == 2 ** 63 - 1


def _sizes(groups):
    return np.bincount(np.asarray(groups))


def test_uniform_capacity_group_sizes():
    assert set(_sizes(lite.capacity_groups([1 / 64] * 64, 8))) == {8}
    s = _sizes(lite.capacity_groups([np.float32(1 / 1024)] * 1024, 102))
    assert len(s) == 102 and sorted(s.tolist()) == [10] * 98 + [11] * 4
    s = _sizes(lite.capacity_groups([np.float32(1 / 32768)] * 32768, 3277))
    assert len(s) == 3277 and sorted(s.tolist()) == [9] * 2 + [10] * 3275


def _scan_groups(v, K):
    # The same rule written as scans instead of a walk: t(p) counts the
    # thresholds crossed before p; a group may open at most once per token;
    # and token p can be no earlier than group K - N + p.
    n = len(v)
    V = [math.floor(float(x) * 2 ** 40) for x in v]
    W = sum(V)
    out, cum, low = [], 0, None
    for p in range(n):
        if p == 0:
            t = 0
        else:
            t = min(K - 1, (K * cum) // W) if W > 0 else K - 1
        low = t - p if low is None else min(low, t - p)
        out.append(max(K - n + p, p + low))
        cum += V[p]
    return out


@pytest.mark.parametrize("seed", range(300))
def test_walk_equals_scan(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 60))
    K = int(rng.integers(1, n + 1))
    kind = seed % 4
    if kind == 0:
        v = rng.random(n)
    elif kind == 1:
        v = rng.random(n) ** 6                    # a few heavy tokens
    elif kind == 2:
        v = np.where(rng.random(n) < 0.3, 0.0, rng.random(n))
        v[0] += 1e-3
    else:
        v = np.ones(n)
    v = (v / v.sum()).astype(np.float32)
    g = lite.capacity_groups(v.tolist(), K)
    assert g == _scan_groups(v.tolist(), K)
    # Exactly K non-empty contiguous groups, in order.
    assert g[0] == 0 and g[-1] == K - 1
    assert all(b - a in (0, 1) for a, b in zip(g, g[1:]))


def test_all_capacity_below_resolution():
    # Every V_j rounds to 0 (W = 0): each threshold counts as reached, so the
    # walk opens a group at every token until the last group.
    v = [np.float32(1e-15)] * 10
    g = lite.capacity_groups(v, 4)
    assert g == [0, 1, 2, 3, 3, 3, 3, 3, 3, 3]
    assert g == _scan_groups(v, 4)


def test_group_mass_near_one_over_k():
    rng = np.random.default_rng(7)
    v = rng.random(5000) + 0.5
    v = (v / v.sum()).astype(np.float32)
    K = 200
    g = np.array(lite.capacity_groups(v.tolist(), K))
    mass = np.bincount(g, weights=v.astype(np.float64), minlength=K)
    assert np.all(np.abs(mass - 1.0 / K) <= v.max() + 1e-9)


def test_toy_hand_values(toy):
    F, X, tau, v = toy["F"], toy["X"], toy["tau"], toy["v"]
    # h = 4 m: every token in voxel (0,0,0).  Grid step 4/256 m, so x = 1 m ->
    # q = 64 -> key 64 interleaved = 2^18 = 262144; y = 2 m -> q = 128 -> 2^22.
    out = lite.lite_ref(F, X, tau, v, 2, h=4.0)
    assert out["keys"].tolist() == [0, 262144, 4194304, 6291456]
    assert out["group"].tolist() == [0, 0, 1, 1]
    # Maxima over the two groups' pairs: M_f from tokens 2,3 (1 - 1/sqrt 2),
    # M_x = 2 (tokens 2,3), M_tau = 1.
    assert np.allclose(out["maxima"], (1 - 1 / math.sqrt(2), 2.0, 1.0), rtol=1e-14)
    assert np.allclose(out["cost"], [0.186805, 0.436805, 0.5, 0.75], atol=6e-7)
    assert out["selected"].tolist() == [0, 2]
    assert out["objective"] == pytest.approx(0.686805, abs=6e-7)
    # h = 1 m: tokens 2 and 3 are two voxels apart in x, so their pair costs
    # c0 = 3; every evaluated pair has equal features (M_f = 0).
    out = lite.lite_ref(F, X, tau, v, 2, h=1.0)
    assert out["keys"].tolist() == [0, 16777216, 268435456, 402653184]
    assert out["maxima"] == (0.0, 1.0, 1.0)
    assert np.allclose(out["cost"], [0.25, 0.5, 0.75, 0.75], atol=1e-15)
    assert out["selected"].tolist() == [0, 2]          # tie 2 vs 3 -> smaller index
    assert out["objective"] == pytest.approx(1.0, abs=1e-15)


def test_one_group_one_voxel_is_full_weighted_medoid():
    s = make_scene("n1024_d256_f32", 5)
    s = subscene(s, np.arange(0, 1024, 13))
    F = fst.widen_features(s.feats, s.dtype)
    out = lite.lite_ref(F, s.pos, s.frame, s.capacity, 1, h=1000.0)
    C, m = fst.fst_cost_ref(F, s.pos, s.frame)
    assert np.allclose(out["maxima"], m, rtol=1e-14)
    w = s.capacity.astype(np.float64)
    cost = C @ w
    assert np.allclose(out["cost"], cost, rtol=1e-12)
    assert out["selected"][0] == int(np.argmin(cost))


def test_costs_agree_with_full_cost_on_evaluated_pairs():
    s = make_scene("n4096_d1152", 1)
    s = subscene(s, np.arange(0, 4096, 23))
    F = fst.widen_features(s.feats, s.dtype)
    K = 20
    out = lite.lite_ref(F, s.pos, s.frame, s.capacity, K, h=0.5)
    C, _ = fst.fst_cost_ref(F, s.pos, s.frame, maxima=out["maxima"])
    vox = out["voxel"]
    adj = np.all(np.abs(vox[:, None, :] - vox[None, :, :]) <= 1, axis=2)
    same = out["group"][:, None] == out["group"][None, :]
    Cl = np.where(adj, C, 3.0)
    w = s.capacity.astype(np.float64)
    expect = np.where(same, Cl, 0.0) @ w
    assert np.allclose(out["cost"], expect, rtol=1e-12)


def test_block_lp_closed_form():
    # Groups with exactly 1/K capacity: the block-constrained optimal plan is
    # P_qj = v_j (Eq. 19-20), so the LP optimum equals the Lite objective.
    s = make_scene("n1024_d256_f32", 2)
    s = subscene(s, np.arange(0, 1024, 64))            # 16 tokens
    v = np.full(16, 1 / 16, np.float32)
    F = fst.widen_features(s.feats, s.dtype)
    K = 4
    out = lite.lite_ref(F, s.pos, s.frame, v, K, h=1000.0)
    assert np.bincount(out["group"]).tolist() == [4, 4, 4, 4]
    C, _ = fst.fst_cost_ref(F, s.pos, s.frame, maxima=out["maxima"])
    val, P = ot.block_ot_lp(C[out["selected"]], np.full(K, 1 / K), v.astype(np.float64),
                            out["group"])
    assert val == pytest.approx(out["objective"], rel=1e-9)
    # Any other prototype choice costs at least as much.
    for q in range(K):
        for t in np.nonzero(out["group"] == q)[0]:
            alt = out["selected"].copy()
            alt[q] = t
            other, _ = ot.block_ot_lp(C[alt], np.full(K, 1 / K), v.astype(np.float64), out["group"])
            assert other >= val - 1e-9

"""Greedy parity on the whole workloads (Sec. 3.5, Eq. 15-16).

Every form of coverprune_sgs_select (dense sweeps; the incremental form's rows
and compact schedules) runs the full budget of the 4096-, 8192- and
16384-token workloads (K = 410, 1229, 1638), seeds 0 and 1, and each
trajectory is replayed step by step against the float64 oracle:

  same cost   the oracle's cost, rounded once to float32, drives the GPU
              greedy; the oracle evaluates exact gains on the same values.
              A pick may differ from the oracle's own choice only where the
              two gains lie within 1e-6 (relative) of each other.
  end to end  the GPU's own cost (coverprune_fst_cost) drives the GPU greedy;
              the oracle evaluates gains on its own float64 cost.  The
              allowance adds the cost error propagated into both gains.

The replay keeps stale upper bounds on every candidate's gain (gains only
shrink), so it evaluates exactly the candidates that could beat the pick and
finishes in seconds at full size.
"""
import gc

import numpy as np
import pytest

from scenes import to_device
from tests import parity

torch = pytest.importorskip("torch")
pytestmark = [pytest.mark.gpu, pytest.mark.slow]

C0 = 3.0
MODES = ["dense", "rows", "compact"]
KINDS = ["same_cost", "end_to_end"]
FULL = [("n4096_d1152", 0), ("n4096_d1152", 1), ("n8192_d3584", 0), ("n8192_d3584", 1),
        ("n16384_d3584", 0), ("n16384_d3584", 1)]
# Grouped by scene, so that each scene's costs are built once.
CASES = [(cfg, seed, kind, mode) for cfg, seed in FULL for kind in KINDS for mode in MODES]

_CACHE = {}


def _cp():
    import paper_2608_13226_amd as cp
    return cp


def _host(r):
    return (r.selected.cpu().numpy(), r.gain.cpu().numpy(), r.objective.cpu().numpy(), r.assign.cpu().numpy())


def _scene_case(cfg, seed):
    key = (cfg, seed)
    if key in _CACHE:
        return _CACHE[key]
    _CACHE.clear()
    gc.collect()
    torch.cuda.empty_cache()
    print(f"building {cfg} seed {seed}", flush=True)
    cp = _cp()
    s = parity.workload_scene(cfg, seed)
    C_ref, maxima = parity.oracle_cost_full(s)                  # float64, source-major
    t = to_device(s)
    runs = {}
    # Same cost: the oracle's cost rounded once to float32, target-major on the GPU.
    C32 = C_ref.astype(np.float32)
    cost = torch.from_numpy(C32).cuda().t().contiguous()
    for mode in MODES:
        print(f"  same-cost greedy {mode}", flush=True)
        r = cp.sgs_select(cost, t["capacity"], s.k, c0=C0, incremental=mode != "dense", compact=mode == "compact")
        torch.cuda.synchronize()
        runs[("same_cost", mode)] = _host(r)
    # End to end: the GPU's own cost.
    print("  fst cost", flush=True)
    cost, m_gpu = cp.fst_cost(t["feats"], t["pos"], t["frame"])
    for mode in MODES:
        print(f"  end-to-end greedy {mode}", flush=True)
        r = cp.sgs_select(cost, t["capacity"], s.k, c0=C0, incremental=mode != "dense", compact=mode == "compact")
        torch.cuda.synchronize()
        runs[("end_to_end", mode)] = _host(r)
    C_gpu = cost.t().contiguous().cpu().numpy()                  # source-major float32
    m_gpu = m_gpu.cpu().numpy()
    del cost, t
    torch.cuda.empty_cache()
    _CACHE[key] = dict(scene=s, C_ref=C_ref, maxima=maxima, C32=C32, C_gpu=C_gpu, m_gpu=m_gpu, runs=runs,
                       replays={})
    return _CACHE[key]


def _oracle_assign(C_src, sel, c0):
    """For every target the earliest pick that covers it most cheaply, -1
    while no pick costs less than c0."""
    rows = np.asarray(C_src[np.asarray(sel, np.int64)], np.float64)
    first = np.argmin(rows, axis=0)
    best = rows[first, np.arange(rows.shape[1])]
    return np.where(best < c0, np.asarray(sel)[first], -1)


@pytest.mark.parametrize("cfg,seed,kind,mode", CASES)
def test_full_workload_greedy(cfg, seed, kind, mode):
    c = _scene_case(cfg, seed)
    s = c["scene"]
    sel, gain, obj, assign = c["runs"][(kind, mode)]
    print(f"sgs full {cfg} seed={seed} n={s.n} k={s.k} {kind} {mode}", flush=True)
    parity.check_trajectory_invariants(sel, gain, obj, s.capacity, C0, s.k, s.n)
    if mode == "compact":
        # The incremental form's two schedules sum the same fixed-point terms
        # over the same block partition: equal bit for bit.
        for x, y in zip(c["runs"][(kind, "rows")], (sel, gain, obj, assign)):
            assert np.array_equal(x, y)
    rkey = (kind, sel.tobytes())
    if rkey not in c["replays"]:
        if kind == "same_cost":
            c["replays"][rkey] = parity.lazy_replay(c["C32"], s.capacity, C0, sel)
        else:
            c["replays"][rkey] = parity.lazy_replay(c["C_ref"], s.capacity, C0, sel, alt=c["C_gpu"])
    ties, g_or, o_or, near = c["replays"][rkey]
    print(f"  near-tie steps: {[(x['step'], x['pick'], x['oracle'], x['gain'], x['oracle_gain']) for x in near]}",
          flush=True)
    if kind == "same_cost":
        # Same float32 values on both sides: gains differ only by the float32
        # difference b - C and the fixed-point grid; objectives sum exact terms.
        assert np.allclose(gain, g_or, rtol=1e-6, atol=1e-12)
        assert np.allclose(obj, o_or, rtol=1e-9, atol=1e-12)
        assert np.array_equal(assign, _oracle_assign(c["C32"], sel, C0))
    else:
        # The GPU's cost within the cost tolerance of the oracle's, everywhere.
        err = np.abs(c["C_gpu"] - c["C_ref"])
        assert np.all(err <= parity.COST_RTOL * np.abs(c["C_ref"]) + parity.COST_ATOL), f"max err {err.max()}"
        # |gain under one cost - gain under the other| <= sum_j v_j (|db_j| + |dC_j|).
        gain_err = 2.0 * float(err.max()) * float(np.sum(s.capacity, dtype=np.float64))
        del err
        m = c["maxima"]
        assert abs(c["m_gpu"][0] - m[0]) <= 1e-5 * m[0] and abs(c["m_gpu"][1] - m[1]) <= 1e-6 * m[1]
        assert c["m_gpu"][2] == m[2]
        # The GPU's objectives are its own cost's; the oracle's along the same
        # picks differ by the cost error only.
        assert np.allclose(obj, o_or, rtol=1e-4, atol=1e-9)
        assert np.all(np.abs(gain - g_or) <= 1e-6 * np.abs(g_or) + gain_err + 1e-12)

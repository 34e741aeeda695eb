"""Failure handling on the GPU, forced from the host: launches whose bounded
waits give up, and the binding's optional data checks.

COVERPRUNE_TEST_ABORT=1 starts every persistent launch with its abort flag
raised and a zero poll limit, so each block leaves at its first unmet wait;
every kernel still exits normally, the outputs are marked (selected = -1)
and the binding's check raises.  The same workspace then serves a normal
call, whose result must equal a fresh one."""
import numpy as np
import pytest

from scenes import to_device
from tests import parity

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _cp():
    import paper_2608_13226_amd as cp
    return cp


@pytest.fixture(scope="module")
def case():
    s = parity.sample_scene("n4096_d1152", 700, 3, salt=7000)
    C32 = parity.oracle_cost(s)[0].astype(np.float32)
    t = to_device(s)
    t["cost"] = torch.from_numpy(np.ascontiguousarray(C32.T)).cuda()
    return s, t


def _same(a, b):
    for x, y in zip((a.selected, a.gain, a.objective, a.assign), (b.selected, b.gain, b.objective, b.assign)):
        assert torch.equal(x, y)


@pytest.mark.parametrize("mode", ["dense", "rows", "compact"])
def test_greedy_that_gives_up(case, mode, monkeypatch):
    s, t = case
    cp = _cp()
    inc, compact = mode != "dense", mode == "compact"
    flags = (cp.CP_SGS_INCREMENTAL | (cp.CP_SGS_COMPACT if compact else 0)) if inc else cp.CP_SGS_DENSE
    ws = torch.empty(cp.library().coverprune_sgs_workspace(s.n, 70, flags), dtype=torch.uint8, device="cuda")
    print(f"greedy abort path {mode}", flush=True)
    monkeypatch.setenv("COVERPRUNE_TEST_ABORT", "1")
    r = cp.sgs_select(t["cost"], t["capacity"], 70, c0=3.0, workspace=ws, incremental=inc, compact=compact)
    torch.cuda.synchronize()
    assert bool((r.selected == -1).all())
    with pytest.raises(cp.CoverPruneError, match="gave up"):
        r.check()
    monkeypatch.delenv("COVERPRUNE_TEST_ABORT")
    again = cp.sgs_select(t["cost"], t["capacity"], 70, c0=3.0, workspace=ws, incremental=inc, compact=compact,
                          check=True)
    fresh = cp.sgs_select(t["cost"], t["capacity"], 70, c0=3.0, incremental=inc, compact=compact, check=True)
    _same(again, fresh)
    parity.replay_greedy(parity.oracle_cost(s)[0].astype(np.float32), s.capacity, 3.0, again.selected.cpu().numpy())


def test_batch_that_gives_up(case, monkeypatch):
    s, t = case
    cp = _cp()
    print("batch abort path", flush=True)
    monkeypatch.setenv("COVERPRUNE_TEST_ABORT", "1")
    rs = cp.sgs_select_batch([t["cost"], t["cost"]], [t["capacity"], t["capacity"]], [50, 20], c0=3.0)
    torch.cuda.synchronize()
    for r in rs:
        assert bool((r.selected == -1).all())
        with pytest.raises(cp.CoverPruneError):
            r.check()
    monkeypatch.delenv("COVERPRUNE_TEST_ABORT")
    rs = cp.sgs_select_batch([t["cost"], t["cost"]], [t["capacity"], t["capacity"]], [50, 20], c0=3.0, check=True)
    alone = cp.sgs_select(t["cost"], t["capacity"], 50, c0=3.0, incremental=True, check=True)
    assert torch.equal(rs[0].selected, alone.selected)


def test_local_greedy_that_gives_up(case, monkeypatch):
    s, t = case
    cp = _cp()
    nbr = cp.knn(t["pos"], 32)
    print("local greedy abort path", flush=True)
    monkeypatch.setenv("COVERPRUNE_TEST_ABORT", "1")
    r = cp.sgs_local_select(t["cost"], t["capacity"], nbr, 40, c0=3.0)
    torch.cuda.synchronize()
    assert bool((r.selected == -1).all())
    with pytest.raises(cp.CoverPruneError):
        r.check()
    monkeypatch.delenv("COVERPRUNE_TEST_ABORT")
    a = cp.sgs_local_select(t["cost"], t["capacity"], nbr, 40, c0=3.0, check=True)
    b = cp.sgs_local_select(t["cost"], t["capacity"], nbr, 40, c0=3.0, check=True)
    _same(a, b)


def test_lite_has_no_waits_to_give_up(case, monkeypatch):
    # Lite's kernels are ordinary launches whose blocks never wait for each
    # other: with every bounded wait set to give up at once, the call still
    # returns its normal result.
    s, t = case
    cp = _cp()
    ws = torch.empty(cp.library().coverprune_lite_workspace(s.n, s.dim, 70, cp.CP_BF16), dtype=torch.uint8,
                     device="cuda")
    print("lite under COVERPRUNE_TEST_ABORT", flush=True)
    monkeypatch.setenv("COVERPRUNE_TEST_ABORT", "1")
    a = cp.lite_select(t["feats"], t["pos"], t["frame"], t["capacity"], 70, workspace=ws, token_cost=True, check=True)
    monkeypatch.delenv("COVERPRUNE_TEST_ABORT")
    ref = parity.lite_reference(s, 70, h=0.25)
    parity.assert_lite_close(a.selected.cpu().numpy(), a.group.cpu().numpy(), float(a.objective.cpu()[0]), ref,
                             a.token_cost.cpu().numpy())
    b = cp.lite_select(t["feats"], t["pos"], t["frame"], t["capacity"], 70, workspace=ws, token_cost=True, check=True)
    assert torch.equal(a.selected, b.selected) and torch.equal(a.group, b.group)


def test_debug_mode_checks_the_data(case, monkeypatch):
    s, t = case
    cp = _cp()
    print("COVERPRUNE_DEBUG data checks", flush=True)
    monkeypatch.setenv("COVERPRUNE_DEBUG", "1")
    feats = t["feats"].clone()
    feats[5, 7] = float("nan")
    with pytest.raises(cp.CoverPruneError, match="features"):
        cp.fst_cost(feats, t["pos"], t["frame"])
    pos = t["pos"].clone()
    pos[3, 1] = float("inf")
    with pytest.raises(cp.CoverPruneError, match="positions"):
        cp.lite_select(t["feats"], pos, t["frame"], t["capacity"], 10)
    neg = t["capacity"].clone()
    neg[0] = -1e-3
    with pytest.raises(cp.CoverPruneError, match=">= 0"):
        cp.sgs_select(t["cost"], neg, 10, c0=3.0)
    with pytest.raises(cp.CoverPruneError, match="positive sum"):
        cp.sgs_select(t["cost"], torch.zeros_like(t["capacity"]), 10, c0=3.0, incremental=True)
    bad = t["cost"].clone()
    bad[2, 9] = float("nan")
    with pytest.raises(cp.CoverPruneError, match="cost"):
        cp.sgs_select(bad, t["capacity"], 10, c0=3.0)
    # Valid data passes, and the call comes back checked.
    cost, _ = cp.fst_cost(t["feats"], t["pos"], t["frame"])
    r = cp.sgs_select(cost, t["capacity"], 10, incremental=True)
    assert int(r.selected.min()) >= 0

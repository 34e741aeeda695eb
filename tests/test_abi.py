"""The C-ABI library on the CPU: it loads, exports every symbol the header
declares, and rejects bad arguments on the host before launching anything.
No call here reaches a kernel, so no GPU is needed."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "coverprune.h")

OK, INVALID, UNSUPPORTED, WORKSPACE = 0, 1, 2, 3
FAKE = ctypes.c_void_p(0x1000)          # aligned, never dereferenced by the host checks


@pytest.fixture(scope="module")
def lib():
    import paper_2608_13226_amd as cp
    if not os.path.exists(cp.library_path()):
        from paper_2608_13226_amd import build
        build.build()
    return cp.library()


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(coverprune_\w+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    names = _declared()
    assert {"coverprune_fst_cost", "coverprune_sgs_select", "coverprune_lite_select"} <= set(names)
    for name in names:
        assert hasattr(lib, name), f"{name} declared in the header but not exported"


def test_version_and_status_strings(lib):
    assert lib.coverprune_abi_version() == 2
    for code, text in [(0, b"ok"), (1, b"invalid argument"), (2, b"unsupported"),
                       (3, b"workspace too small"), (4, b"HIP runtime error")]:
        assert lib.coverprune_status_string(code) == text
    assert lib.coverprune_status_string(99) == b"unknown status"


def test_workspace_queries(lib):
    assert lib.coverprune_fst_cost_workspace(0, 8, 1) == 0
    assert lib.coverprune_fst_cost_workspace(16384, 3584, 1) >= 16384 * 4
    a = lib.coverprune_sgs_workspace(1024, 102, 0)
    b = lib.coverprune_sgs_workspace(16384, 1638, 0)
    # the compact incremental schedule needs far less than the dense form's
    # partial gains; the rows schedule adds the source-major copy of the cost
    c = lib.coverprune_sgs_workspace(16384, 1638, 3)
    assert 16384 * 16 <= c < b
    r = lib.coverprune_sgs_workspace(16384, 1638, 1)
    # ... and, up to n = 16384, the early steps' per-block partial sums
    # (256 blocks of n + 1 columns rounded up to 64, 8 bytes each) and the
    # hand-over between launches (gains, chosen flags, best costs: 13 bytes
    # per token, and 1280 bytes); past 128 picks also the candidate lists
    # (256 pairs of 16 bytes per token)
    early = 256 * 16448 * 8
    ho = 16384 * 13 + 1280
    assert r == c + 16384 * 16384 * 4 + early + 16384 * 256 * 16 + ho
    assert lib.coverprune_sgs_workspace(16384, 128, 1) == (lib.coverprune_sgs_workspace(16384, 128, 3)
                                                           + 16384 * 16384 * 4 + early + ho)
    # ... up to n = 32768 (rows padded to 256 targets; 16 blocks at n = 1000);
    # beyond it the compact one
    assert lib.coverprune_sgs_workspace(1000, 100, 1) == (lib.coverprune_sgs_workspace(1000, 100, 3)
                                                          + 1000 * 1024 * 4 + 16 * 1024 * 8
                                                          + 8192 + 1024 + 4096 + 1280)
    assert lib.coverprune_sgs_workspace(32769, 100, 1) == lib.coverprune_sgs_workspace(32769, 100, 3)
    assert lib.coverprune_sgs_workspace(16384, 1638, 2) == 0      # compact alone is not a form
    assert 0 < a < b
    # at least two radix key buffers, two token buffers and the packed voxel words
    assert lib.coverprune_lite_workspace(32768, 3584, 3277, 1) >= 32768 * 40


def _w(lf=1.0, lx=1.0, lt=1.0, kappa=10.0):
    import paper_2608_13226_amd as cp
    return cp._Weights(lf, lx, lt, kappa)


def _fst(lib, **kw):
    a = dict(feats=FAKE, dtype=1, n=64, d=64, pos=FAKE, frame=FAKE, w=_w(), cost=FAKE, maxima=None,
             ws=FAKE, ws_bytes=1 << 30, stream=None)
    a.update(kw)
    return lib.coverprune_fst_cost(a["feats"], a["dtype"], a["n"], a["d"], a["pos"], a["frame"], a["w"],
                                   a["cost"], a["maxima"], a["ws"], a["ws_bytes"], a["stream"])


@pytest.mark.parametrize("kw,code", [
    (dict(n=0), INVALID), (dict(n=-5), INVALID), (dict(n=1 << 19), INVALID),
    (dict(d=0), INVALID), (dict(d=12), UNSUPPORTED), (dict(dtype=0, d=6), UNSUPPORTED),
    (dict(dtype=7), UNSUPPORTED), (dict(feats=None), INVALID), (dict(pos=None), INVALID),
    (dict(frame=None), INVALID), (dict(cost=None), INVALID),
    (dict(feats=ctypes.c_void_p(0x1004)), INVALID),
    (dict(w=_w(lf=-1.0)), INVALID), (dict(w=_w(kappa=float("nan"))), INVALID),
    (dict(ws=None), WORKSPACE), (dict(ws_bytes=16), WORKSPACE),
])
def test_fst_cost_rejects(lib, kw, code):
    assert _fst(lib, **kw) == code
    assert lib.coverprune_last_error() != b""


def _sgs(lib, **kw):
    a = dict(cost=FAKE, n=64, v=FAKE, k=8, c0=3.0, flags=0, sel=FAKE, gain=None, obj=None, assign=None,
             ws=FAKE, ws_bytes=1 << 30, stream=None)
    a.update(kw)
    return lib.coverprune_sgs_select(a["cost"], a["n"], a["v"], a["k"], a["c0"], a["flags"], a["sel"],
                                     a["gain"], a["obj"], a["assign"], a["ws"], a["ws_bytes"], a["stream"])


@pytest.mark.parametrize("kw,code", [
    (dict(n=0), INVALID), (dict(k=0), INVALID), (dict(k=65), INVALID), (dict(k=-1), INVALID),
    (dict(c0=float("inf")), INVALID), (dict(flags=7), UNSUPPORTED), (dict(flags=2), UNSUPPORTED),
    (dict(flags=3, ws_bytes=100), WORKSPACE), (dict(flags=1, ws_bytes=64 * 16 + 1024), WORKSPACE),
    (dict(cost=None), INVALID),
    (dict(v=None), INVALID), (dict(sel=None), INVALID), (dict(ws=None), WORKSPACE),
    (dict(ws_bytes=100), WORKSPACE), (dict(ws=ctypes.c_void_p(0x1008)), WORKSPACE),
])
def test_sgs_rejects(lib, kw, code):
    assert _sgs(lib, **kw) == code


def _lite(lib, **kw):
    a = dict(feats=FAKE, dtype=1, n=64, d=64, pos=FAKE, frame=FAKE, v=FAKE, k=8, w=_w(), h=0.25,
             sel=FAKE, group=None, obj=None, tcost=None, ws=FAKE, ws_bytes=1 << 30, stream=None)
    a.update(kw)
    return lib.coverprune_lite_select(a["feats"], a["dtype"], a["n"], a["d"], a["pos"], a["frame"], a["v"],
                                      a["k"], a["w"], a["h"], a["sel"], a["group"], a["obj"], a["tcost"], a["ws"],
                                      a["ws_bytes"], a["stream"])


@pytest.mark.parametrize("kw,code", [
    (dict(n=0), INVALID), (dict(k=0), INVALID), (dict(k=65), INVALID), (dict(h=0.0), INVALID),
    (dict(h=-1.0), INVALID), (dict(h=float("inf")), INVALID), (dict(d=4), UNSUPPORTED),
    (dict(v=None), INVALID), (dict(sel=None), INVALID), (dict(pos=None), INVALID),
    (dict(ws=None), WORKSPACE), (dict(ws_bytes=64), WORKSPACE), (dict(w=_w(lt=-2.0)), INVALID),
])
def test_lite_rejects(lib, kw, code):
    assert _lite(lib, **kw) == code


@pytest.mark.parametrize("kw,code", [
    (dict(n=0), INVALID), (dict(n=32769), INVALID), (dict(k=0), INVALID), (dict(k=65), INVALID),
    (dict(cost=None), INVALID), (dict(cap=None), INVALID), (dict(sel=None), INVALID),
    (dict(c0=float("nan")), INVALID), (dict(cost=ctypes.c_void_p(0x1004)), INVALID),
])
def test_sgs_noalloc_rejects(lib, kw, code):
    # Host checks only: every rejection happens before the device is touched.
    a = dict(cost=FAKE, n=64, cap=FAKE, k=8, c0=3.0, sel=FAKE)
    a.update(kw)
    assert lib.coverprune_sgs_select_noalloc(a["cost"], a["n"], a["cap"], a["k"], ctypes.c_float(a["c0"]), a["sel"],
                                             None, None, None, None) == code


@pytest.mark.parametrize("kw,code", [
    (dict(n=0), INVALID), (dict(row_len=100), INVALID), (dict(row_len=0), INVALID),
    (dict(row_len=32768 + 256), INVALID), (dict(rounds=0), INVALID), (dict(rows=None), INVALID),
    (dict(ws=None), WORKSPACE), (dict(ws_bytes=16), WORKSPACE),
])
def test_step_floor_rejects(lib, kw, code):
    a = dict(rows=FAKE, n=64, row_len=256, rounds=10, read=1, ws=FAKE, ws_bytes=1 << 20)
    a.update(kw)
    assert lib.coverprune_step_floor(a["rows"], a["n"], a["row_len"], a["rounds"], a["read"], a["ws"], a["ws_bytes"],
                                     None) == code


def test_uncovered_cost_is_the_largest_cost(lib):
    # c0 = (lambda_f + lambda_x) + lambda_tau in float arithmetic: every term of
    # Eq. 8 is at most its weight once normalised.
    import paper_2608_13226_amd as cp
    assert lib.coverprune_uncovered_cost(cp._Weights(1.0, 1.0, 1.0, 10.0)) == 3.0
    assert lib.coverprune_uncovered_cost(cp._Weights(0.5, 2.0, 0.25, 0.0)) == 2.75
    x = lib.coverprune_uncovered_cost(cp._Weights(0.1, 0.2, 0.3, 1.0))
    f = ctypes.c_float
    assert x == f(f(f(0.1).value + f(0.2).value).value + f(0.3).value).value
    assert cp.uncovered_cost((1.0, 1.0, 1.0)) == 3.0


def test_binding_rejects_a_library_of_another_abi(monkeypatch):
    import paper_2608_13226_amd as cp
    monkeypatch.setattr(cp, "_lib", None)
    monkeypatch.setattr(cp, "ABI_VERSION", 1)
    with pytest.raises(cp.CoverPruneError, match="ABI"):
        cp.library()


def test_binding_needs_the_library(monkeypatch, tmp_path):
    # The Python layer never falls back to anything else: a missing library is an error.
    import paper_2608_13226_amd as cp
    monkeypatch.setattr(cp, "_lib", None)
    monkeypatch.setattr(cp, "library_path", lambda: str(tmp_path / "missing.so"))
    with pytest.raises(cp.CoverPruneError):
        cp.library()


def test_local_workspace_query(lib):
    assert lib.coverprune_sgs_local_workspace(0, 8) == 0
    # exchange slots, one objective part per block and step, the transposed cost
    ws = lib.coverprune_sgs_local_workspace(16384, 1638)
    assert 16384 * 16384 * 4 + 1638 * 256 * 8 <= ws < 16384 * 16384 * 4 + 1638 * 256 * 8 + (1 << 22)
    assert lib.coverprune_sgs_local_workspace(1000, 10) >= 1000 * 1024 * 4


def _knn(lib, **kw):
    a = dict(pos=FAKE, n=64, g=8, out=FAKE, stream=None)
    a.update(kw)
    return lib.coverprune_knn(a["pos"], a["n"], a["g"], a["out"], a["stream"])


@pytest.mark.parametrize("kw,code", [
    (dict(n=0), INVALID), (dict(n=32769, g=8), INVALID), (dict(g=0), INVALID), (dict(g=65), INVALID),
    (dict(n=4096, g=1025), INVALID), (dict(pos=None), INVALID), (dict(out=None), INVALID),
])
def test_knn_rejects(lib, kw, code):
    assert _knn(lib, **kw) == code
    assert lib.coverprune_last_error() != b""


def _local(lib, **kw):
    a = dict(cost=FAKE, n=64, v=FAKE, nbr=FAKE, g=8, k=8, c0=3.0, sel=FAKE, gain=None, obj=None, assign=None,
             ws=FAKE, ws_bytes=1 << 30, stream=None)
    a.update(kw)
    return lib.coverprune_sgs_local_select(a["cost"], a["n"], a["v"], a["nbr"], a["g"], a["k"], a["c0"], a["sel"],
                                           a["gain"], a["obj"], a["assign"], a["ws"], a["ws_bytes"], a["stream"])


@pytest.mark.parametrize("kw,code", [
    (dict(n=0), INVALID), (dict(n=16385), INVALID), (dict(g=0), INVALID), (dict(g=65), INVALID),
    (dict(n=1024, g=129), INVALID), (dict(k=0), INVALID), (dict(k=65), INVALID),
    (dict(c0=float("nan")), INVALID), (dict(cost=None), INVALID), (dict(v=None), INVALID),
    (dict(nbr=None), INVALID), (dict(sel=None), INVALID), (dict(cost=ctypes.c_void_p(0x1004)), INVALID),
    (dict(ws=None), WORKSPACE), (dict(ws_bytes=100), WORKSPACE),
])
def test_sgs_local_rejects(lib, kw, code):
    assert _local(lib, **kw) == code


def _cw(af=1.0, ax=1.0, at=1.0):
    import paper_2608_13226_amd as cp
    return cp._CapWeights(af, ax, at)


def test_capacity_workspace_query(lib):
    assert lib.coverprune_fst_capacity_workspace(1, 1) == 0
    assert lib.coverprune_fst_capacity_workspace(64, 64) == 0
    assert lib.coverprune_fst_capacity_workspace(16384, 16) >= 16384 * (4 * 17 + 24 * 16)


def _cap(lib, **kw):
    a = dict(feats=FAKE, dtype=1, n=64, d=64, pos=FAKE, frame=FAKE, nn=8, alpha=_cw(), v=FAKE, r=None,
             ws=FAKE, ws_bytes=1 << 30, stream=None)
    a.update(kw)
    return lib.coverprune_fst_capacity(a["feats"], a["dtype"], a["n"], a["d"], a["pos"], a["frame"], a["nn"],
                                       a["alpha"], a["v"], a["r"], a["ws"], a["ws_bytes"], a["stream"])


@pytest.mark.parametrize("kw,code", [
    (dict(n=1, nn=1), INVALID), (dict(n=32769), INVALID), (dict(nn=0), INVALID), (dict(nn=64), INVALID),
    (dict(n=4096, nn=1024), INVALID), (dict(d=12), UNSUPPORTED), (dict(feats=None), INVALID),
    (dict(pos=None), INVALID), (dict(frame=None), INVALID), (dict(v=None), INVALID),
    (dict(alpha=_cw(af=-1.0)), INVALID), (dict(alpha=_cw(at=float("inf"))), INVALID),
    (dict(ws=None), WORKSPACE), (dict(ws_bytes=1000), WORKSPACE),
])
def test_capacity_rejects(lib, kw, code):
    assert _cap(lib, **kw) == code


def test_literal_workspace_query(lib):
    assert lib.coverprune_sgs_literal_workspace(0, 1) == 0
    assert lib.coverprune_sgs_literal_workspace(10, 11) == 0
    assert lib.coverprune_sgs_literal_workspace(16384, 1638) >= 16384 * 1640 * 8


def _lit(lib, **kw):
    a = dict(cost=FAKE, n=64, v=FAKE, k=8, eps=0.05, rounds=10, follow=None, sel=FAKE, score=None, resid=None,
             obj=None, ws=FAKE, ws_bytes=1 << 30, stream=None)
    a.update(kw)
    return lib.coverprune_sgs_literal_select(a["cost"], a["n"], a["v"], a["k"], a["eps"], a["rounds"], a["follow"],
                                             a["sel"], a["score"], a["resid"], a["obj"], a["ws"], a["ws_bytes"],
                                             a["stream"])


@pytest.mark.parametrize("kw,code", [
    (dict(n=0), INVALID), (dict(k=0), INVALID), (dict(k=65), INVALID), (dict(n=8192, k=4097), INVALID),
    (dict(eps=0.0), INVALID), (dict(eps=-1.0), INVALID), (dict(eps=float("nan")), INVALID),
    (dict(rounds=0), INVALID), (dict(rounds=1000001), INVALID), (dict(cost=None), INVALID),
    (dict(v=None), INVALID), (dict(sel=None), INVALID), (dict(ws=None), WORKSPACE), (dict(ws_bytes=64), WORKSPACE),
])
def test_literal_rejects(lib, kw, code):
    assert _lit(lib, **kw) == code


def _scenes(count, **kw):
    import paper_2608_13226_amd as cp
    arr = (cp._SgsScene * max(count, 1))()
    for s in range(count):
        a = dict(cost=0x1000, capacity=0x1000, n=64, k=8, c0=3.0, selected=0x1000, step_gain=None,
                 step_objective=None, assign=None)
        if s == count - 1:
            a.update(kw)
        arr[s] = cp._SgsScene(a["cost"], a["capacity"], a["n"], a["k"], a["c0"], a["selected"], a["step_gain"],
                              a["step_objective"], a["assign"])
    return arr


def test_batch_workspace_is_the_sum_of_the_scenes(lib):
    for flags in (1, 3):
        one = lib.coverprune_sgs_workspace(64, 8, flags)
        assert lib.coverprune_sgs_batch_workspace(_scenes(3), 3, flags) == 3 * one
        assert lib.coverprune_sgs_batch_workspace(_scenes(3), 17, flags) == 0
    assert lib.coverprune_sgs_batch_workspace(_scenes(3), 3, 0) == 0
    assert lib.coverprune_sgs_batch_workspace(_scenes(3), 3, 2) == 0


@pytest.mark.parametrize("count,kw,code", [
    (0, {}, INVALID), (17, {}, INVALID), (3, dict(n=0), INVALID), (3, dict(k=0), INVALID), (3, dict(k=65), INVALID),
    (2, dict(c0=float("inf")), INVALID), (2, dict(cost=None), INVALID), (2, dict(capacity=None), INVALID),
    (2, dict(selected=None), INVALID), (2, dict(cost=0x1004), INVALID),
])
def test_batch_rejects(lib, count, kw, code):
    arr = _scenes(max(count, 1), **kw) if count <= 16 else _scenes(16)
    assert lib.coverprune_sgs_select_batch(arr, count, 1, FAKE, 1 << 30, None) == code
    assert lib.coverprune_last_error() != b""


def test_batch_rejects_small_workspace(lib):
    assert lib.coverprune_sgs_select_batch(_scenes(2), 2, 1, FAKE, 64, None) == WORKSPACE
    assert lib.coverprune_sgs_select_batch(_scenes(2), 2, 1, None, 1 << 30, None) == WORKSPACE
    assert lib.coverprune_sgs_select_batch(None, 2, 1, FAKE, 1 << 30, None) == INVALID


@pytest.mark.parametrize("flags", [0, 2, 4, 5, 7])
def test_batch_rejects_flags(lib, flags):
    assert lib.coverprune_sgs_select_batch(_scenes(2), 2, flags, FAKE, 1 << 30, None) == UNSUPPORTED

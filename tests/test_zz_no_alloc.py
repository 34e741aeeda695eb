"""coverprune_sgs_select_noalloc through the C-ABI: the greedy with its
scratch in the library's static device array gives, call after call, what
coverprune_sgs_select gives with a workspace in the same schedule
(CP_SGS_INCREMENTAL | CP_SGS_COMPACT): the same kernels, so equal bit for
bit, and a valid greedy trajectory by the oracle."""
import ctypes

import numpy as np
import pytest

from tests import parity

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _lib():
    import paper_2608_13226_amd as cp
    lib = cp.library()
    lib.coverprune_sgs_select_noalloc.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64,
                                                  ctypes.c_float] + [ctypes.c_void_p] * 5
    lib.coverprune_sgs_select_noalloc.restype = ctypes.c_int
    return cp, lib


def _p(t):
    return ctypes.c_void_p(t.data_ptr())


def _noalloc(cp, lib, cost, cap, k, c0):
    n = cost.shape[0]
    out = cp.SgsResult(torch.empty(k, dtype=torch.int32, device="cuda"),
                       torch.empty(k, dtype=torch.float64, device="cuda"),
                       torch.empty(k, dtype=torch.float64, device="cuda"),
                       torch.empty(n, dtype=torch.int32, device="cuda"))
    st = lib.coverprune_sgs_select_noalloc(_p(cost), n, _p(cap), k, c0, _p(out.selected), _p(out.gain),
                                           _p(out.objective), _p(out.assign),
                                           ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == 0, lib.coverprune_last_error().decode()
    return out


def test_noalloc_matches_the_workspace_form_twice():
    cp, lib = _lib()
    # Two calls in a row on the same scratch, the second on a smaller scene.
    for cfg, n, k, seed in [("n4096_d1152", 3000, 300, 0), ("n1024_d256_f32", 700, 70, 1)]:
        s = parity.sample_scene(cfg, n, seed, salt=9000)
        C32 = parity.oracle_cost(s)[0].astype(np.float32)
        cost = torch.from_numpy(np.ascontiguousarray(C32.T)).cuda()
        cap = torch.from_numpy(s.capacity).cuda()
        print(f"noalloc greedy {cfg} n={s.n} k={k}", flush=True)
        got = _noalloc(cp, lib, cost, cap, k, 3.0)
        ref = cp.sgs_select(cost, cap, k, c0=3.0, incremental=True, compact=True)
        torch.cuda.synchronize()
        for x, y in zip((got.selected, got.gain, got.objective, got.assign),
                        (ref.selected, ref.gain, ref.objective, ref.assign)):
            assert torch.equal(x, y)
        sel = got.selected.cpu().numpy()
        ties, g_or, o_or = parity.replay_greedy(C32, s.capacity, 3.0, sel)
        assert np.allclose(got.gain.cpu().numpy(), g_or, rtol=1e-6, atol=1e-12)
        assert np.allclose(got.objective.cpu().numpy(), o_or, rtol=1e-9, atol=1e-12)


def test_noalloc_rejects_scenes_beyond_its_scratch():
    cp, lib = _lib()
    fake = ctypes.c_void_p(0x1000)
    st = lib.coverprune_sgs_select_noalloc(fake, 40000, fake, 10, 3.0, fake, None, None, None, None)
    assert st == 1 and b"scratch" in lib.coverprune_last_error()

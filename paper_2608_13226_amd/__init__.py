"""CoverPrune's hot path on AMD Instinct MI355X.

Python binding of ``libcoverprune.so`` (C-ABI in include/coverprune.h).  The
functions here only check and marshal torch tensors: every step runs in the
library's HIP kernels.  Tensors must live on the current GPU; work is
enqueued on torch's current stream and nothing synchronises the host, with
two exceptions that the caller asks for:

* ``check=True`` on a selection call (or ``result.check()`` later)
  synchronises the stream and raises CoverPruneError when the launch's
  bounded waits gave up (the library then marks ``selected`` with -1);
* ``COVERPRUNE_DEBUG=1`` in the environment validates the data before every
  call (finite features, positions and costs; capacities finite, >= 0, with
  a positive sum), which the library itself does not read for validity, and
  then checks every selection as ``check=True`` does.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

import torch

__all__ = ["fst_cost", "fst_capacity", "prune", "sgs_select", "sgs_select_batch", "sgs_literal_select", "knn",
           "sgs_local_select", "lite_select", "uncovered_cost", "step_floor", "library", "library_path", "CoverPruneError",
           "DEFAULT_KAPPA"]

HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_NAME = "libcoverprune.so"

# The paper leaves kappa open (Sec. 3.3 only requires kappa > 0).
DEFAULT_KAPPA = 10.0
ABI_VERSION = 2

CP_F32, CP_BF16 = 0, 1
CP_SGS_DENSE = 0
CP_SGS_INCREMENTAL = 1
CP_SGS_COMPACT = 2


class CoverPruneError(RuntimeError):
    pass


def _debug() -> bool:
    return os.environ.get("COVERPRUNE_DEBUG", "") == "1"


def _require(ok: bool, msg: str) -> None:
    if not ok:
        raise CoverPruneError(f"COVERPRUNE_DEBUG: {msg}")


def _debug_features(feats, pos, frame) -> None:
    _require(bool(torch.isfinite(feats).all()), "features hold NaN or infinite values")
    _require(bool(torch.isfinite(pos).all()), "positions hold NaN or infinite values")


def _debug_capacity(capacity) -> None:
    _require(bool(torch.isfinite(capacity).all()), "capacities hold NaN or infinite values")
    _require(bool((capacity >= 0).all()), "capacities must be >= 0")
    _require(float(capacity.double().sum()) > 0.0, "capacities must have a positive sum")


def _debug_cost(cost) -> None:
    _require(bool(torch.isfinite(cost).all()), "the cost holds NaN or infinite values")


def _check_selected(selected: torch.Tensor, stream, what: str) -> None:
    """Synchronise ``stream`` and raise when the launch gave up (-1 picks)."""
    s = torch.cuda.current_stream() if stream is None else stream
    s.synchronize()
    if selected.numel() and int(selected[0].item()) < 0:
        raise CoverPruneError(f"{what}: the launch gave up waiting (bounded wait exceeded); "
                              f"selected holds -1")


class _Weights(ctypes.Structure):
    _fields_ = [("lambda_f", ctypes.c_float), ("lambda_x", ctypes.c_float),
                ("lambda_tau", ctypes.c_float), ("kappa", ctypes.c_float)]


class _SgsScene(ctypes.Structure):
    _fields_ = [("cost", ctypes.c_void_p), ("capacity", ctypes.c_void_p), ("n", ctypes.c_int64),
                ("k", ctypes.c_int64), ("c0", ctypes.c_float), ("selected", ctypes.c_void_p),
                ("step_gain", ctypes.c_void_p), ("step_objective", ctypes.c_void_p), ("assign", ctypes.c_void_p)]


class _CapWeights(ctypes.Structure):
    _fields_ = [("alpha_f", ctypes.c_float), ("alpha_x", ctypes.c_float), ("alpha_tau", ctypes.c_float)]


_lib = None


def library_path() -> str:
    return os.path.join(HERE, _LIB_NAME)


def library() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    path = library_path()
    if not os.path.exists(path):
        raise CoverPruneError(f"{path} is missing: build it with `python -m paper_2608_13226_amd.build`")
    lib = ctypes.CDLL(path)
    i64, sz, vp, u32 = ctypes.c_int64, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_uint32
    st = ctypes.c_int
    lib.coverprune_fst_cost_workspace.argtypes = [i64, i64, ctypes.c_int]
    lib.coverprune_fst_cost_workspace.restype = sz
    lib.coverprune_fst_cost.argtypes = [vp, ctypes.c_int, i64, i64, vp, vp, _Weights, vp, vp, vp, sz, vp]
    lib.coverprune_fst_cost.restype = st
    lib.coverprune_sgs_workspace.argtypes = [i64, i64, ctypes.c_uint32]
    lib.coverprune_sgs_workspace.restype = sz
    lib.coverprune_prune_workspace.argtypes = [i64, i64, i64, ctypes.c_int]
    lib.coverprune_prune_workspace.restype = sz
    lib.coverprune_prune.argtypes = [vp, ctypes.c_int, i64, i64, vp, vp, _Weights, vp, i64, ctypes.c_float,
                                     vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.coverprune_prune.restype = st
    lib.coverprune_sgs_select.argtypes = [vp, i64, vp, i64, ctypes.c_float, u32, vp, vp, vp, vp, vp, sz, vp]
    lib.coverprune_sgs_select.restype = st
    lib.coverprune_fst_capacity_workspace.argtypes = [i64, i64]
    lib.coverprune_fst_capacity_workspace.restype = sz
    lib.coverprune_fst_capacity.argtypes = [vp, ctypes.c_int, i64, i64, vp, vp, i64, _CapWeights, vp, vp, vp, sz,
                                            vp]
    lib.coverprune_fst_capacity.restype = st
    lib.coverprune_sgs_batch_workspace.argtypes = [ctypes.POINTER(_SgsScene), ctypes.c_int32, ctypes.c_uint32]
    lib.coverprune_sgs_batch_workspace.restype = sz
    lib.coverprune_sgs_select_batch.argtypes = [ctypes.POINTER(_SgsScene), ctypes.c_int32, ctypes.c_uint32, vp, sz, vp]
    lib.coverprune_sgs_select_batch.restype = st
    lib.coverprune_sgs_literal_workspace.argtypes = [i64, i64]
    lib.coverprune_sgs_literal_workspace.restype = sz
    lib.coverprune_sgs_literal_select.argtypes = [vp, i64, vp, i64, ctypes.c_float, ctypes.c_int32, vp, vp, vp, vp,
                                                  vp, vp, sz, vp]
    lib.coverprune_sgs_literal_select.restype = st
    lib.coverprune_knn.argtypes = [vp, i64, i64, vp, vp]
    lib.coverprune_knn.restype = st
    lib.coverprune_sgs_local_workspace.argtypes = [i64, i64]
    lib.coverprune_sgs_local_workspace.restype = sz
    lib.coverprune_sgs_local_select.argtypes = [vp, i64, vp, vp, i64, i64, ctypes.c_float, vp, vp, vp, vp, vp,
                                                sz, vp]
    lib.coverprune_sgs_local_select.restype = st
    lib.coverprune_lite_workspace.argtypes = [i64, i64, i64, ctypes.c_int]
    lib.coverprune_lite_workspace.restype = sz
    lib.coverprune_lite_select.argtypes = [vp, ctypes.c_int, i64, i64, vp, vp, vp, i64, _Weights,
                                           ctypes.c_float, vp, vp, vp, vp, vp, sz, vp]
    lib.coverprune_lite_select.restype = st
    lib.coverprune_status_string.argtypes = [st]
    lib.coverprune_status_string.restype = ctypes.c_char_p
    lib.coverprune_last_error.argtypes = []
    lib.coverprune_last_error.restype = ctypes.c_char_p
    lib.coverprune_abi_version.argtypes = []
    lib.coverprune_abi_version.restype = ctypes.c_int
    lib.coverprune_sgs_select_noalloc.argtypes = [vp, i64, vp, i64, ctypes.c_float, vp, vp, vp, vp, vp]
    lib.coverprune_sgs_select_noalloc.restype = st
    lib.coverprune_step_floor_workspace.argtypes = []
    lib.coverprune_step_floor_workspace.restype = sz
    lib.coverprune_step_floor.argtypes = [vp, i64, i64, ctypes.c_int32, ctypes.c_int32, vp, sz, vp]
    lib.coverprune_step_floor.restype = st
    lib.coverprune_uncovered_cost.argtypes = [_Weights]
    lib.coverprune_uncovered_cost.restype = ctypes.c_float
    if lib.coverprune_abi_version() != ABI_VERSION:
        raise CoverPruneError(f"{path} has ABI {lib.coverprune_abi_version()}, this binding needs {ABI_VERSION}: "
                              f"rebuild it")
    _lib = lib
    return lib


def _check(status: int) -> None:
    if status != 0:
        lib = library()
        raise CoverPruneError(f"{lib.coverprune_status_string(status).decode()}: "
                              f"{lib.coverprune_last_error().decode()}")


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _need(t: torch.Tensor, name: str, dtype, shape, device) -> None:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if t.device != device:
        raise ValueError(f"{name} must be on {device}, got {t.device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _feature_dtype(feats: torch.Tensor) -> int:
    if feats.dtype == torch.bfloat16:
        return CP_BF16
    if feats.dtype == torch.float32:
        return CP_F32
    raise TypeError(f"features must be bfloat16 or float32, got {feats.dtype}")


def _workspace(nbytes: int, device) -> torch.Tensor:
    return torch.empty(max(int(nbytes), 16), dtype=torch.uint8, device=device)


def _weights(weights, kappa) -> _Weights:
    lf, lx, lt = (float(w) for w in weights)
    return _Weights(lf, lx, lt, float(kappa))


def uncovered_cost(weights=(1.0, 1.0, 1.0)) -> float:
    """c0 of the greedy for a cost made with ``weights``: the largest value
    the cost can take (coverprune_uncovered_cost)."""
    return float(library().coverprune_uncovered_cost(_weights(weights, 0.0)))


def fst_cost(feats: torch.Tensor, pos: torch.Tensor, frame: torch.Tensor,
             weights=(1.0, 1.0, 1.0), kappa: float = DEFAULT_KAPPA,
             out: Optional[torch.Tensor] = None, maxima: Optional[torch.Tensor] = None,
             workspace: Optional[torch.Tensor] = None, stream=None):
    """FST transport cost (Sec. 3.3, Eq. 7-8), target-major: out[t, s] = C(s, t).

    Returns (cost [n, n] float32, maxima [3] float32 = M_f, M_x, M_tau)."""
    lib = library()
    n, d = feats.shape
    dev = feats.device
    dt = _feature_dtype(feats)
    _need(feats, "feats", feats.dtype, (n, d), dev)
    _need(pos, "pos", torch.float32, (n, 3), dev)
    _need(frame, "frame", torch.int32, (n,), dev)
    if _debug():
        _debug_features(feats, pos, frame)
    if out is None:
        out = torch.empty((n, n), dtype=torch.float32, device=dev)
    _need(out, "out", torch.float32, (n, n), dev)
    if maxima is None:
        maxima = torch.empty(3, dtype=torch.float32, device=dev)
    _need(maxima, "maxima", torch.float32, (3,), dev)
    need = lib.coverprune_fst_cost_workspace(n, d, dt)
    if workspace is None:
        workspace = _workspace(need, dev)
    _check(lib.coverprune_fst_cost(_ptr(feats), dt, n, d, _ptr(pos), _ptr(frame), _weights(weights, kappa),
                                   _ptr(out), _ptr(maxima), _ptr(workspace), workspace.numel(),
                                   _stream(stream)))
    return out, maxima


def fst_capacity(feats: torch.Tensor, pos: torch.Tensor, frame: torch.Tensor, n_nb: int,
                 alpha=(1.0, 1.0, 1.0), out: Optional[torch.Tensor] = None,
                 score: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None, stream=None):
    """FST capacity (Sec. 3.4, Eq. 9-10) from each token's n_nb nearest other
    tokens.  Returns (v [n] float32 summing to 1, r [n] float64 scores)."""
    lib = library()
    n, d = feats.shape
    dev = feats.device
    dt = _feature_dtype(feats)
    _need(feats, "feats", feats.dtype, (n, d), dev)
    _need(pos, "pos", torch.float32, (n, 3), dev)
    _need(frame, "frame", torch.int32, (n,), dev)
    if _debug():
        _debug_features(feats, pos, frame)
    if out is None:
        out = torch.empty(n, dtype=torch.float32, device=dev)
    _need(out, "out", torch.float32, (n,), dev)
    if score is None:
        score = torch.empty(n, dtype=torch.float64, device=dev)
    _need(score, "score", torch.float64, (n,), dev)
    need = lib.coverprune_fst_capacity_workspace(n, int(n_nb))
    if workspace is None:
        workspace = _workspace(need, dev)
    a_f, a_x, a_t = (float(a) for a in alpha)
    _check(lib.coverprune_fst_capacity(_ptr(feats), dt, n, d, _ptr(pos), _ptr(frame), int(n_nb),
                                       _CapWeights(a_f, a_x, a_t), _ptr(out), _ptr(score), _ptr(workspace),
                                       workspace.numel(), _stream(stream)))
    return out, score


@dataclass
class SgsResult:
    selected: torch.Tensor     # [k] int32, greedy order
    gain: torch.Tensor         # [k] float64
    objective: torch.Tensor    # [k] float64, L(S) after each step
    assign: torch.Tensor       # [n] int32

    def check(self, stream=None) -> "SgsResult":
        """Synchronise and raise CoverPruneError if the launch gave up."""
        _check_selected(self.selected, stream, "greedy selection")
        return self


def _c0(c0, weights) -> float:
    return uncovered_cost(weights) if c0 is None else float(c0)


def sgs_select(cost: torch.Tensor, capacity: torch.Tensor, k: int, c0: Optional[float] = None,
               weights=(1.0, 1.0, 1.0), workspace: Optional[torch.Tensor] = None,
               stream=None, incremental: bool = False, compact: bool = False, check: bool = False) -> SgsResult:
    """Greedy selection of k tokens over a target-major cost (Sec. 3.5, Eq. 11-16).
    c0 defaults to coverprune_uncovered_cost(weights), the largest value C
    takes.  incremental=True runs the same greedy with gains updated from the
    rows whose best cost drops (CP_SGS_INCREMENTAL) instead of full sweeps;
    compact=True (with incremental) picks the small-workspace schedule.
    check=True synchronises and raises if the launch gave up."""
    lib = library()
    n = cost.shape[0]
    dev = cost.device
    _need(cost, "cost", torch.float32, (n, n), dev)
    _need(capacity, "capacity", torch.float32, (n,), dev)
    if _debug():
        _debug_cost(cost)
        _debug_capacity(capacity)
    c0 = _c0(c0, weights)
    sel = torch.empty(int(k), dtype=torch.int32, device=dev)
    gain = torch.empty(int(k), dtype=torch.float64, device=dev)
    obj = torch.empty(int(k), dtype=torch.float64, device=dev)
    assign = torch.empty(n, dtype=torch.int32, device=dev)
    if compact and not incremental:
        raise ValueError("compact=True needs incremental=True")
    flags = (CP_SGS_INCREMENTAL | (CP_SGS_COMPACT if compact else 0)) if incremental else CP_SGS_DENSE
    need = lib.coverprune_sgs_workspace(n, int(k), flags)
    if workspace is None:
        workspace = _workspace(need, dev)
    _check(lib.coverprune_sgs_select(_ptr(cost), n, _ptr(capacity), int(k), float(c0), flags,
                                     _ptr(sel), _ptr(gain), _ptr(obj), _ptr(assign), _ptr(workspace),
                                     workspace.numel(), _stream(stream)))
    r = SgsResult(sel, gain, obj, assign)
    return r.check(stream) if (check or _debug()) else r


def prune(feats: torch.Tensor, pos: torch.Tensor, frame: torch.Tensor, capacity: torch.Tensor, k: int,
          c0: Optional[float] = None, weights=(1.0, 1.0, 1.0), kappa: float = DEFAULT_KAPPA,
          out: Optional[torch.Tensor] = None, maxima: Optional[torch.Tensor] = None,
          workspace: Optional[torch.Tensor] = None, stream=None, check: bool = False):
    """The whole prune of one scene (Sec. 3): the FST cost and the
    incremental greedy in one call (coverprune_prune), the same result as
    fst_cost followed by sgs_select(incremental=True).  c0 defaults to
    coverprune_uncovered_cost(weights).  Returns (cost, maxima, SgsResult)."""
    lib = library()
    n, d = feats.shape
    dev = feats.device
    dt = _feature_dtype(feats)
    _need(feats, "feats", feats.dtype, (n, d), dev)
    _need(pos, "pos", torch.float32, (n, 3), dev)
    _need(frame, "frame", torch.int32, (n,), dev)
    _need(capacity, "capacity", torch.float32, (n,), dev)
    if _debug():
        _debug_features(feats, pos, frame)
        _debug_capacity(capacity)
    if out is None:
        out = torch.empty((n, n), dtype=torch.float32, device=dev)
    _need(out, "out", torch.float32, (n, n), dev)
    if maxima is None:
        maxima = torch.empty(3, dtype=torch.float32, device=dev)
    _need(maxima, "maxima", torch.float32, (3,), dev)
    c0 = _c0(c0, weights)
    sel = torch.empty(int(k), dtype=torch.int32, device=dev)
    gain = torch.empty(int(k), dtype=torch.float64, device=dev)
    obj = torch.empty(int(k), dtype=torch.float64, device=dev)
    assign = torch.empty(n, dtype=torch.int32, device=dev)
    need = lib.coverprune_prune_workspace(n, d, int(k), dt)
    if workspace is None:
        workspace = _workspace(need, dev)
    _check(lib.coverprune_prune(_ptr(feats), dt, n, d, _ptr(pos), _ptr(frame), _weights(weights, kappa),
                                _ptr(capacity), int(k), float(c0), _ptr(out), _ptr(maxima), _ptr(sel), _ptr(gain),
                                _ptr(obj), _ptr(assign), _ptr(workspace), workspace.numel(), _stream(stream)))
    r = SgsResult(sel, gain, obj, assign)
    return out, maxima, (r.check(stream) if (check or _debug()) else r)


def sgs_select_batch(costs, capacities, ks, c0: Optional[float] = None, weights=(1.0, 1.0, 1.0),
                     workspace: Optional[torch.Tensor] = None, stream=None, compact: bool = False,
                     check: bool = False):
    """The incremental greedy of several scenes (lists of target-major costs,
    capacities and budgets) in one launch.  Returns one SgsResult per scene.
    compact=True picks the small-workspace schedule; check as for sgs_select."""
    lib = library()
    count = len(costs)
    if not (len(capacities) == len(ks) == count):
        raise ValueError("costs, capacities and ks must have the same length")
    c0 = _c0(c0, weights)
    arr = (_SgsScene * max(count, 1))()
    out = []
    for s, (cost, cap, k) in enumerate(zip(costs, capacities, ks)):
        n = cost.shape[0]
        dev = cost.device
        _need(cost, f"costs[{s}]", torch.float32, (n, n), dev)
        _need(cap, f"capacities[{s}]", torch.float32, (n,), dev)
        if _debug():
            _debug_cost(cost)
            _debug_capacity(cap)
        r = SgsResult(torch.empty(int(k), dtype=torch.int32, device=dev),
                      torch.empty(int(k), dtype=torch.float64, device=dev),
                      torch.empty(int(k), dtype=torch.float64, device=dev),
                      torch.empty(n, dtype=torch.int32, device=dev))
        arr[s] = _SgsScene(cost.data_ptr(), cap.data_ptr(), n, int(k), float(c0), r.selected.data_ptr(),
                           r.gain.data_ptr(), r.objective.data_ptr(), r.assign.data_ptr())
        out.append(r)
    flags = CP_SGS_INCREMENTAL | (CP_SGS_COMPACT if compact else 0)
    need = lib.coverprune_sgs_batch_workspace(arr, count, flags)
    if workspace is None:
        workspace = _workspace(need, costs[0].device if count else None)
    _check(lib.coverprune_sgs_select_batch(arr, count, flags, _ptr(workspace), workspace.numel(),
                                           _stream(stream)))
    if check or _debug():
        for r in out:
            r.check(stream)
    return out


@dataclass
class LiteralResult:
    selected: torch.Tensor     # [k] int32, greedy order
    score: torch.Tensor        # [k] float64, score of each pick
    residual: torch.Tensor     # [k] float64, residual mass before each pick
    objective: torch.Tensor    # [1] float64, transport cost of the final plan


def sgs_literal_select(cost: torch.Tensor, capacity: torch.Tensor, k: int, epsilon: float = 0.05,
                       rounds: int = 100, follow: Optional[torch.Tensor] = None, steps: bool = True,
                       workspace: Optional[torch.Tensor] = None, stream=None) -> LiteralResult:
    """The greedy with each step's entropic semi-relaxed transport solved as
    written (Sec. 3.5, Eq. 11-15).  follow: [k] int32 picks to replay instead
    of the argmin; with steps=False (and follow given) only the final plan is
    solved and score/residual are left empty."""
    lib = library()
    n = cost.shape[0]
    dev = cost.device
    _need(cost, "cost", torch.float32, (n, n), dev)
    _need(capacity, "capacity", torch.float32, (n,), dev)
    if follow is not None:
        _need(follow, "follow", torch.int32, (int(k),), dev)
    sel = torch.empty(int(k), dtype=torch.int32, device=dev)
    score = torch.empty(int(k), dtype=torch.float64, device=dev)
    resid = torch.empty(int(k), dtype=torch.float64, device=dev)
    obj = torch.empty(1, dtype=torch.float64, device=dev)
    need = lib.coverprune_sgs_literal_workspace(n, int(k))
    if workspace is None:
        workspace = _workspace(need, dev)
    keep = steps or follow is None
    _check(lib.coverprune_sgs_literal_select(_ptr(cost), n, _ptr(capacity), int(k), float(epsilon), int(rounds),
                                             _ptr(follow), _ptr(sel), _ptr(score) if keep else None,
                                             _ptr(resid) if keep else None, _ptr(obj), _ptr(workspace),
                                             workspace.numel(), _stream(stream)))
    return LiteralResult(sel, score, resid, obj)


def step_floor(rows: torch.Tensor, rounds: int, read_rows: bool = True, workspace: Optional[torch.Tensor] = None,
               stream=None) -> None:
    """Enqueue `rounds` rounds of the greedy's candidate exchange, each
    followed (read_rows) by the read of the row of ``rows`` [n, row_len]
    float32 that the round's winner names: the latency floor of a greedy
    step (coverprune_step_floor).  Time it with events on the stream."""
    lib = library()
    if rows.dim() != 2:
        raise ValueError("rows must be [n, row_len]")
    _need(rows, "rows", torch.float32, tuple(rows.shape), rows.device)
    if workspace is None:
        workspace = _workspace(lib.coverprune_step_floor_workspace(), rows.device)
    _check(lib.coverprune_step_floor(_ptr(rows), rows.shape[0], rows.shape[1], int(rounds), int(bool(read_rows)),
                                     _ptr(workspace), workspace.numel(), _stream(stream)))


def knn(pos: torch.Tensor, g: int, out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """The g tokens nearest to every token in 3D (Sec. 3.5, Eq. 13): row t of
    the [n, g] int32 result lists them by (distance, index), t included."""
    lib = library()
    n = pos.shape[0]
    dev = pos.device
    _need(pos, "pos", torch.float32, (n, 3), dev)
    if out is None:
        out = torch.empty((n, int(g)), dtype=torch.int32, device=dev)
    _need(out, "out", torch.int32, (n, int(g)), dev)
    _check(lib.coverprune_knn(_ptr(pos), n, int(g), _ptr(out), _stream(stream)))
    return out


def sgs_local_select(cost: torch.Tensor, capacity: torch.Tensor, neighbours: torch.Tensor, k: int,
                     c0: Optional[float] = None, weights=(1.0, 1.0, 1.0),
                     workspace: Optional[torch.Tensor] = None, stream=None, check: bool = False) -> SgsResult:
    """Greedy selection with each candidate's gain over its neighbour row only
    (Sec. 3.5, Eq. 13); neighbours is an [n, g] int32 table such as knn()
    returns.  c0 and check as for sgs_select."""
    lib = library()
    n = cost.shape[0]
    dev = cost.device
    _need(cost, "cost", torch.float32, (n, n), dev)
    _need(capacity, "capacity", torch.float32, (n,), dev)
    if neighbours.dim() != 2:
        raise ValueError("neighbours must be an [n, g] table")
    g = neighbours.shape[1]
    _need(neighbours, "neighbours", torch.int32, (n, g), dev)
    if _debug():
        _debug_cost(cost)
        _debug_capacity(capacity)
    c0 = _c0(c0, weights)
    sel = torch.empty(int(k), dtype=torch.int32, device=dev)
    gain = torch.empty(int(k), dtype=torch.float64, device=dev)
    obj = torch.empty(int(k), dtype=torch.float64, device=dev)
    assign = torch.empty(n, dtype=torch.int32, device=dev)
    need = lib.coverprune_sgs_local_workspace(n, int(k))
    if workspace is None:
        workspace = _workspace(need, dev)
    _check(lib.coverprune_sgs_local_select(_ptr(cost), n, _ptr(capacity), _ptr(neighbours), g, int(k), float(c0),
                                           _ptr(sel), _ptr(gain), _ptr(obj), _ptr(assign), _ptr(workspace),
                                           workspace.numel(), _stream(stream)))
    r = SgsResult(sel, gain, obj, assign)
    return r.check(stream) if (check or _debug()) else r


@dataclass
class LiteResult:
    selected: torch.Tensor     # [k] int32, prototype of group q at [q]
    group: torch.Tensor        # [n] int32
    objective: torch.Tensor    # [1] float64
    token_cost: torch.Tensor   # [n] float64, each token's cost to its group (Eq. 18)

    def check(self, stream=None) -> "LiteResult":
        """Synchronise and raise CoverPruneError if the launch gave up."""
        _check_selected(self.selected, stream, "Lite selection")
        return self


def lite_select(feats: torch.Tensor, pos: torch.Tensor, frame: torch.Tensor, capacity: torch.Tensor,
                k: int, weights=(1.0, 1.0, 1.0), kappa: float = DEFAULT_KAPPA, voxel_size: float = 0.25,
                workspace: Optional[torch.Tensor] = None, stream=None, token_cost: bool = False,
                check: bool = False) -> LiteResult:
    """CoverPrune-Lite (Sec. 4, Eq. 17-20).  token_cost=True also returns
    every token's cost to its group; check as for sgs_select."""
    lib = library()
    n, d = feats.shape
    dev = feats.device
    dt = _feature_dtype(feats)
    _need(feats, "feats", feats.dtype, (n, d), dev)
    _need(pos, "pos", torch.float32, (n, 3), dev)
    _need(frame, "frame", torch.int32, (n,), dev)
    _need(capacity, "capacity", torch.float32, (n,), dev)
    if _debug():
        _debug_features(feats, pos, frame)
        _debug_capacity(capacity)
    sel = torch.empty(int(k), dtype=torch.int32, device=dev)
    group = torch.empty(n, dtype=torch.int32, device=dev)
    obj = torch.empty(1, dtype=torch.float64, device=dev)
    tc = torch.empty(n if token_cost else 0, dtype=torch.float64, device=dev)
    need = lib.coverprune_lite_workspace(n, d, int(k), dt)
    if workspace is None:
        workspace = _workspace(need, dev)
    _check(lib.coverprune_lite_select(_ptr(feats), dt, n, d, _ptr(pos), _ptr(frame), _ptr(capacity), int(k),
                                      _weights(weights, kappa), float(voxel_size), _ptr(sel), _ptr(group),
                                      _ptr(obj), _ptr(tc) if token_cost else None, _ptr(workspace),
                                      workspace.numel(), _stream(stream)))
    r = LiteResult(sel, group, obj, tc)
    return r.check(stream) if (check or _debug()) else r

"""ctypes binding of libtwinkv.so (C ABI in include/twinkv.h).

Argument marshalling only: torch supplies device memory and the current HIP stream;
every step of the computation runs in the library's HIP kernels.  The library must have
been built (``python -m paper_2608_27128_amd.build``); a missing build raises.

Shapes: keys (n_heads, T, d) or (T, d) with the channel dimension contiguous, bfloat16 or
float32, on a GPU; retained / outputs (n_heads, T).  ``cu_seqlens`` (host sequence of
n_seqs + 1 ints) splits T into sequences; the default is one sequence of length T.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtwinkv.so")

TWINKV_OK = 0
TWINKV_BF16, TWINKV_F32 = 0, 1
OP_NN_SCORES, OP_REPAIR, OP_REPAIR_FROM_SCORES, OP_TWIN_COUNTS, OP_SCORE_EVICT, OP_COMPACT = range(6)
MAX_TAUS = 32
MAX_LEVELS = 4
PROBLEM_OK, PROBLEM_BUDGET_MISMATCH, PROBLEM_NONFINITE = 0, 1, 2

_lib = None

_VP = ctypes.c_void_p
_I = ctypes.c_int
_I64 = ctypes.c_int64
_F = ctypes.c_float
_PI64 = ctypes.POINTER(ctypes.c_int64)

SIGNATURES = {
    "twinkv_workspace_bytes": (_I64, [_I, _I, _I, _I, _I, _PI64]),
    "twinkv_nn_scores": (_I, [_VP, _I, _I, _I, _I, _PI64, _I64, _I64, _VP, _I,
                              _VP, _VP, _VP, _VP, _VP, _VP, _I64, _VP]),
    "twinkv_repair": (_I, [_VP, _I, _I, _I, _I, _PI64, _I64, _I64, _VP, _VP, _PI64, _F, _I, _I, _I,
                           _VP, _VP, _VP, _VP, _VP, _VP, _I64, _VP]),
    "twinkv_repair_from_scores": (_I, [_VP, _VP, _VP, _I, _I, _PI64, _PI64, _F, _I, _I, _VP,
                                       _VP, _I64, _VP]),
    "twinkv_twin_counts": (_I, [_VP, _I, _I, _I, _I, _PI64, _I64, _I64, _F, _I, _VP, _VP, _VP,
                                _I64, _VP]),
    "twinkv_score_evict": (_I, [_VP, _I, _I, _I, _I, _PI64, _I64, _I64, _PI64, _F, _I, _I, _I,
                                _VP, _VP, _VP, _VP, _VP, _I64, _VP]),
    "twinkv_prevalence": (_I, [_VP, _I, _I, _PI64, ctypes.POINTER(ctypes.c_float), _I, _VP, _VP,
                               _I64, _VP]),
    "twinkv_select_topk": (_I, [_VP, _I, _I, _PI64, _PI64, _I, _I, _VP, _VP, _VP, _I64, _VP]),
    "twinkv_nn_scores_levels": (_I, [_VP, _I, _I, _I, _I, _PI64, _I64, _I64, _VP, _I, _I, _VP,
                                     _VP, _VP, _VP, _VP, _VP, _I64, _VP]),
    "twinkv_levels_workspace_bytes": (_I64, [_I, _I, _I, _I, _PI64, _I, _I]),
    "twinkv_compact": (_I, [_VP, _VP, _I, _I, _I, _I, _PI64, _I64, _I64, _I64, _I64, _VP, _PI64,
                            _VP, _VP, _VP, _VP, _VP, _I64, _VP]),
    "twinkv_status_string": (ctypes.c_char_p, [_I]),
    "twinkv_version": (_I, []),
    "twinkv_profile_sim_events": (None, [_VP, _VP]),
}


class TwinKVError(RuntimeError):
    def __init__(self, fn: str, code: int):
        super().__init__(f"{fn} failed: {status_string(code)} (code {code})")
        self.code = code


def lib() -> ctypes.CDLL:
    """The loaded library (loads it on first use; raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2608_27128_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def status_string(code: int) -> str:
    return lib().twinkv_status_string(int(code)).decode()


def version() -> int:
    return int(lib().twinkv_version())


def _i64_array(values) -> ctypes.Array:
    arr = np.ascontiguousarray(np.asarray(values, dtype=np.int64))
    return (ctypes.c_int64 * len(arr))(*arr.tolist())


def workspace_bytes(op: int, dtype: int, d: int, n_heads: int, cu_seqlens) -> int:
    cu = _i64_array(cu_seqlens)
    n = int(lib().twinkv_workspace_bytes(op, dtype, d, n_heads, len(cu) - 1, cu))
    if n < 0:
        raise TwinKVError("twinkv_workspace_bytes", -n)
    return n


def levels_workspace_bytes(dtype: int, d: int, n_heads: int, cu_seqlens, n_levels: int,
                           want_all: bool) -> int:
    cu = _i64_array(cu_seqlens)
    n = int(lib().twinkv_levels_workspace_bytes(dtype, d, n_heads, len(cu) - 1, cu,
                                                int(n_levels), 1 if want_all else 0))
    if n < 0:
        raise TwinKVError("twinkv_levels_workspace_bytes", -n)
    return n


def _event_handle(e):
    if e is None:
        return None
    if isinstance(e, ctypes.c_void_p):
        return e.value
    return int(e)


def profile_sim_events(start=None, stop=None) -> None:
    """Record two hipEvent_t handles (ints or c_void_p) around the similarity kernel of later
    calls on this thread (None, None stops)."""
    lib().twinkv_profile_sim_events(_event_handle(start), _event_handle(stop))


def _torch():
    import torch
    return torch


def _prep_keys(keys):
    torch = _torch()
    if keys.dim() == 2:
        keys = keys.unsqueeze(0)
    if keys.dim() != 3:
        raise ValueError("keys must be (n_heads, T, d) or (T, d)")
    if not keys.is_cuda:
        raise ValueError("keys must be on a GPU")
    if keys.stride(2) != 1:
        keys = keys.contiguous()
    if keys.dtype == torch.bfloat16:
        dt = TWINKV_BF16
    elif keys.dtype == torch.float32:
        dt = TWINKV_F32
    else:
        raise ValueError(f"unsupported key dtype {keys.dtype}")
    return keys, dt


def _cu(cu_seqlens, T: int):
    return np.array([0, T], dtype=np.int64) if cu_seqlens is None else np.asarray(cu_seqlens, dtype=np.int64)


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(device) -> int:
    torch = _torch()
    return torch.cuda.current_stream(device).cuda_stream


def _mask(x, n_heads, T, device, name):
    torch = _torch()
    if x is None:
        return None
    if x.dim() == 1:
        x = x.unsqueeze(0)
    if tuple(x.shape) != (n_heads, T):
        raise ValueError(f"{name} must have shape ({n_heads}, {T})")
    if x.dtype == torch.bool:
        x = x.to(torch.uint8)
    if x.dtype != torch.uint8:
        raise ValueError(f"{name} must be uint8 or bool")
    if x.device != device:
        raise ValueError(f"{name} must be on {device}")
    return x.contiguous()


def nn_scores(keys, retained=None, w: int = 32, cu_seqlens=None, *, want_arg: bool = True,
              workspace=None) -> dict:
    """Best twin of every token: best_all/arg_all over all keys, best_ret/arg_ret (Eq. 4 b_i(S0))
    over the retained set when ``retained`` is given, and a per-problem status."""
    torch = _torch()
    keys, dt = _prep_keys(keys)
    H, T, d = keys.shape
    dev = keys.device
    cu = _cu(cu_seqlens, T)
    if cu[-1] != T:
        raise ValueError("cu_seqlens[-1] must equal T")
    ret = _mask(retained, H, T, dev, "retained")
    out = {
        "best_all": torch.empty((H, T), dtype=torch.float32, device=dev),
        "arg_all": torch.empty((H, T), dtype=torch.int32, device=dev) if want_arg else None,
        "status": torch.empty((H * (len(cu) - 1),), dtype=torch.int32, device=dev),
    }
    if ret is not None:
        out["best_ret"] = torch.empty((H, T), dtype=torch.float32, device=dev)
        out["arg_ret"] = torch.empty((H, T), dtype=torch.int32, device=dev) if want_arg else None
    nbytes = workspace_bytes(OP_NN_SCORES, dt, d, H, cu)
    ws = workspace if workspace is not None and workspace.numel() >= nbytes else \
        torch.empty((nbytes,), dtype=torch.uint8, device=dev)
    cu_c = _i64_array(cu)
    rc = lib().twinkv_nn_scores(
        keys.data_ptr(), dt, d, H, len(cu) - 1, cu_c, keys.stride(0), keys.stride(1),
        _ptr(ret), int(w), _ptr(out["best_all"]), _ptr(out["arg_all"]),
        _ptr(out.get("best_ret")), _ptr(out.get("arg_ret")), _ptr(out["status"]),
        ws.data_ptr(), ws.numel(), _stream(dev))
    if rc != TWINKV_OK:
        raise TwinKVError("twinkv_nn_scores", rc)
    return {k: v for k, v in out.items() if v is not None}


def nn_scores_levels(keys, level, n_levels: int, w: int = 32, cu_seqlens=None, *,
                     want_all: bool = False, want_arg: bool = True, workspace=None,
                     outputs: Optional[dict] = None) -> dict:
    """b_i(S_k) (Sec. 3.4 Eq. 4) for nested retained sets S_1 within ... within S_L given as a
    level array (n_heads, T) uint8 (k = the smallest set holding the token, 0 = none):
    best_lvl / arg_lvl of shape (n_levels, n_heads, T), and best_all / arg_all when
    ``want_all``.  ``outputs`` may pass back the dict of an earlier call."""
    torch = _torch()
    keys, dt = _prep_keys(keys)
    H, T, d = keys.shape
    dev = keys.device
    cu = _cu(cu_seqlens, T)
    if cu[-1] != T:
        raise ValueError("cu_seqlens[-1] must equal T")
    n_seqs = len(cu) - 1
    lv = _mask(level, H, T, dev, "level")
    if lv is None:
        raise ValueError("level is required")
    if outputs is None:
        out = {
            "best_lvl": torch.empty((n_levels, H, T), dtype=torch.float32, device=dev),
            "arg_lvl": torch.empty((n_levels, H, T), dtype=torch.int32, device=dev) if want_arg else None,
            "best_all": torch.empty((H, T), dtype=torch.float32, device=dev) if want_all else None,
            "arg_all": torch.empty((H, T), dtype=torch.int32, device=dev) if (want_all and want_arg) else None,
            "status": torch.empty((H * n_seqs,), dtype=torch.int32, device=dev),
        }
    else:
        out = dict(outputs)
    cu_c = _i64_array(cu)
    nbytes = levels_workspace_bytes(dt, d, H, cu, n_levels, want_all)
    ws = workspace if workspace is not None and workspace.numel() >= nbytes else \
        torch.empty((nbytes,), dtype=torch.uint8, device=dev)
    rc = lib().twinkv_nn_scores_levels(
        keys.data_ptr(), dt, d, H, n_seqs, cu_c, keys.stride(0), keys.stride(1), lv.data_ptr(),
        int(n_levels), int(w), _ptr(out.get("best_all")), _ptr(out.get("arg_all")),
        out["best_lvl"].data_ptr(), _ptr(out.get("arg_lvl")), _ptr(out["status"]),
        ws.data_ptr(), ws.numel(), _stream(dev))
    if rc != TWINKV_OK:
        raise TwinKVError("twinkv_nn_scores_levels", rc)
    return {k: v for k, v in out.items() if v is not None}


def repair(keys, retained, budget, tau: float, w: int = 32, n_sink: int = 4, n_recent: int = 64,
           cu_seqlens=None, *, want_all: bool = True, want_arg: bool = True, out_mask=None,
           workspace=None, outputs: Optional[dict] = None) -> dict:
    """The repair pass of Sec. 3.4: S1 (uint8 mask), stats (|O|, |D|, m, status) per problem,
    and the scores it was computed from (best_ret = b; best_all/arg_all when want_all).

    ``outputs`` may pass back the dict of an earlier call with the same shapes to reuse its
    buffers; ``out_mask`` may be ``retained`` itself for an in-place update."""
    torch = _torch()
    keys, dt = _prep_keys(keys)
    H, T, d = keys.shape
    dev = keys.device
    cu = _cu(cu_seqlens, T)
    n_seqs = len(cu) - 1
    ret = _mask(retained, H, T, dev, "retained")
    if ret is None:
        raise ValueError("retained is required")
    bud = np.broadcast_to(np.asarray(budget, dtype=np.int64), (n_seqs,)).copy()
    if outputs is None:
        def f32():
            return torch.empty((H, T), dtype=torch.float32, device=dev)

        def i32():
            return torch.empty((H, T), dtype=torch.int32, device=dev)
        out = {
            "s1": torch.empty((H, T), dtype=torch.uint8, device=dev),
            "stats": torch.empty((H * n_seqs, 4), dtype=torch.int32, device=dev),
            "best_ret": f32(),
            "arg_ret": i32() if want_arg else None,
            "best_all": f32() if want_all else None,
            "arg_all": i32() if (want_all and want_arg) else None,
        }
    else:
        out = dict(outputs)
    if out_mask is not None:
        out["s1"] = out_mask
    nbytes = workspace_bytes(OP_REPAIR, dt, d, H, cu)
    ws = workspace if workspace is not None and workspace.numel() >= nbytes else \
        torch.empty((nbytes,), dtype=torch.uint8, device=dev)
    rc = lib().twinkv_repair(
        keys.data_ptr(), dt, d, H, n_seqs, _i64_array(cu), keys.stride(0), keys.stride(1),
        ret.data_ptr(), out["s1"].data_ptr(), _i64_array(bud), float(tau), int(w), int(n_sink),
        int(n_recent), out["stats"].data_ptr(), _ptr(out.get("best_all")), _ptr(out.get("arg_all")),
        _ptr(out.get("best_ret")), _ptr(out.get("arg_ret")), ws.data_ptr(), ws.numel(), _stream(dev))
    if rc != TWINKV_OK:
        raise TwinKVError("twinkv_repair", rc)
    return {k: v for k, v in out.items() if v is not None}


def repair_from_scores(b, retained, budget, tau: float, n_sink: int = 4, n_recent: int = 64,
                       cu_seqlens=None, *, out_mask=None) -> dict:
    """Classification, ranking and swap of Sec. 3.4 from given scores b (n_heads, T) float32."""
    torch = _torch()
    if b.dim() == 1:
        b = b.unsqueeze(0)
    if b.dtype != torch.float32 or not b.is_cuda:
        raise ValueError("b must be a float32 GPU tensor")
    b = b.contiguous()
    H, T = b.shape
    dev = b.device
    cu = _cu(cu_seqlens, T)
    n_seqs = len(cu) - 1
    ret = _mask(retained, H, T, dev, "retained")
    if ret is None:
        raise ValueError("retained is required")
    bud = np.broadcast_to(np.asarray(budget, dtype=np.int64), (n_seqs,)).copy()
    s1 = out_mask if out_mask is not None else torch.empty((H, T), dtype=torch.uint8, device=dev)
    stats = torch.empty((H * n_seqs, 4), dtype=torch.int32, device=dev)
    nbytes = workspace_bytes(OP_REPAIR_FROM_SCORES, 0, 64, H, cu)
    ws = torch.empty((nbytes,), dtype=torch.uint8, device=dev)
    rc = lib().twinkv_repair_from_scores(
        b.data_ptr(), ret.data_ptr(), s1.data_ptr(), H, n_seqs, _i64_array(cu), _i64_array(bud),
        float(tau), int(n_sink), int(n_recent), stats.data_ptr(), ws.data_ptr(), ws.numel(),
        _stream(dev))
    if rc != TWINKV_OK:
        raise TwinKVError("twinkv_repair_from_scores", rc)
    return {"s1": s1, "stats": stats}


def twin_counts(keys, tau: float, w: int = 32, cu_seqlens=None, *, workspace=None) -> dict:
    """Eq. 2 twin counts r_i (int32, (n_heads, T)) and a per-problem status."""
    torch = _torch()
    keys, dt = _prep_keys(keys)
    H, T, d = keys.shape
    dev = keys.device
    cu = _cu(cu_seqlens, T)
    if cu[-1] != T:
        raise ValueError("cu_seqlens[-1] must equal T")
    counts = torch.empty((H, T), dtype=torch.int32, device=dev)
    status = torch.empty((H * (len(cu) - 1),), dtype=torch.int32, device=dev)
    nbytes = workspace_bytes(OP_TWIN_COUNTS, dt, d, H, cu)
    ws = workspace if workspace is not None and workspace.numel() >= nbytes else \
        torch.empty((nbytes,), dtype=torch.uint8, device=dev)
    rc = lib().twinkv_twin_counts(
        keys.data_ptr(), dt, d, H, len(cu) - 1, _i64_array(cu), keys.stride(0), keys.stride(1),
        float(tau), int(w), counts.data_ptr(), status.data_ptr(), ws.data_ptr(), ws.numel(),
        _stream(dev))
    if rc != TWINKV_OK:
        raise TwinKVError("twinkv_twin_counts", rc)
    return {"counts": counts, "status": status}


def score_evict(keys, budget, tau: float, w: int = 32, n_sink: int = 4, n_recent: int = 64,
                cu_seqlens=None, *, want_scores: bool = True, workspace=None,
                outputs: Optional[dict] = None) -> dict:
    """The standalone scorer of Sec. 3.2: counts (Eq. 2), scores (Eq. 3), the kept set of the
    `budget` highest scores (uint8) and per-problem stats {kept, count at cut, status, 0}.
    ``outputs`` may pass back the dict of an earlier call with the same shapes."""
    torch = _torch()
    keys, dt = _prep_keys(keys)
    H, T, d = keys.shape
    dev = keys.device
    cu = _cu(cu_seqlens, T)
    n_seqs = len(cu) - 1
    bud = np.broadcast_to(np.asarray(budget, dtype=np.int64), (n_seqs,)).copy()
    if outputs is None:
        out = {
            "retained": torch.empty((H, T), dtype=torch.uint8, device=dev),
            "counts": torch.empty((H, T), dtype=torch.int32, device=dev),
            "scores": torch.empty((H, T), dtype=torch.float32, device=dev) if want_scores else None,
            "stats": torch.empty((H * n_seqs, 4), dtype=torch.int32, device=dev),
        }
    else:
        out = dict(outputs)
        out.setdefault("scores", None)
    nbytes = workspace_bytes(OP_SCORE_EVICT, dt, d, H, cu)
    ws = workspace if workspace is not None and workspace.numel() >= nbytes else \
        torch.empty((nbytes,), dtype=torch.uint8, device=dev)
    rc = lib().twinkv_score_evict(
        keys.data_ptr(), dt, d, H, n_seqs, _i64_array(cu), keys.stride(0), keys.stride(1),
        _i64_array(bud), float(tau), int(w), int(n_sink), int(n_recent),
        out["retained"].data_ptr(), out["counts"].data_ptr(), _ptr(out["scores"]),
        out["stats"].data_ptr(), ws.data_ptr(), ws.numel(), _stream(dev))
    if rc != TWINKV_OK:
        raise TwinKVError("twinkv_score_evict", rc)
    return {k: v for k, v in out.items() if v is not None}


def select_topk(scores, budget, n_sink: int = 4, n_recent: int = 64, cu_seqlens=None, *,
                workspace=None, outputs: Optional[dict] = None) -> dict:
    """A score-based policy's retained set (Sec. 3.1 / 3.2): per problem the ``budget[s]``
    positions first in the order protected, higher score, lower position (NaN last).
    scores: float32 (n_heads, T) on the GPU.  Returns retained uint8 (n_heads, T) and
    stats int32 (n_heads * n_seqs, 4) = {kept, NaN scores, 0, 0}."""
    torch = _torch()
    if scores.dim() == 1:
        scores = scores.unsqueeze(0)
    if scores.dtype != torch.float32 or not scores.is_cuda:
        raise ValueError("scores must be a float32 GPU tensor")
    scores = scores.contiguous()
    H, T = scores.shape
    dev = scores.device
    cu = _cu(cu_seqlens, T)
    if cu[-1] != T:
        raise ValueError("cu_seqlens[-1] must equal T")
    n_seqs = len(cu) - 1
    bud = np.broadcast_to(np.asarray(budget, dtype=np.int64), (n_seqs,))
    out = outputs if outputs is not None else {
        "retained": torch.empty((H, T), dtype=torch.uint8, device=dev),
        "stats": torch.empty((H * n_seqs, 4), dtype=torch.int32, device=dev),
    }
    nbytes = workspace_bytes(OP_REPAIR_FROM_SCORES, 0, 64, H, cu)
    ws = workspace if workspace is not None and workspace.numel() >= nbytes else \
        torch.empty((nbytes,), dtype=torch.uint8, device=dev)
    rc = lib().twinkv_select_topk(
        scores.data_ptr(), H, n_seqs, _i64_array(cu), _i64_array(bud), int(n_sink),
        int(n_recent), out["retained"].data_ptr(), _ptr(out["stats"]), ws.data_ptr(),
        ws.numel(), _stream(dev))
    if rc != TWINKV_OK:
        raise TwinKVError("twinkv_select_topk", rc)
    return out


def prevalence(best_all, taus, cu_seqlens=None) -> "torch.Tensor":
    """Tokens with at least one twin (best_all > tau) per problem and threshold:
    int32 (n_heads * n_seqs, len(taus))."""
    torch = _torch()
    if best_all.dim() == 1:
        best_all = best_all.unsqueeze(0)
    if best_all.dtype != torch.float32 or not best_all.is_cuda:
        raise ValueError("best_all must be a float32 GPU tensor")
    best_all = best_all.contiguous()
    H, T = best_all.shape
    dev = best_all.device
    cu = _cu(cu_seqlens, T)
    n_seqs = len(cu) - 1
    tv = np.ascontiguousarray(np.asarray(taus, dtype=np.float32))
    out = torch.empty((H * n_seqs, len(tv)), dtype=torch.int32, device=dev)
    nbytes = workspace_bytes(OP_REPAIR_FROM_SCORES, 0, 64, H, cu)
    ws = torch.empty((nbytes,), dtype=torch.uint8, device=dev)
    rc = lib().twinkv_prevalence(
        best_all.data_ptr(), H, n_seqs, _i64_array(cu),
        tv.ctypes.data_as(ctypes.POINTER(ctypes.c_float)), len(tv), out.data_ptr(),
        ws.data_ptr(), ws.numel(), _stream(dev))
    if rc != TWINKV_OK:
        raise TwinKVError("twinkv_prevalence", rc)
    return out


def compact(keys, retained, capacity, values=None, cu_seqlens=None, *, want_pos: bool = True,
            workspace=None, outputs: Optional[dict] = None) -> dict:
    """KV compaction (Sec. 3.1): the rows of the retained positions of every problem, in
    position order, in its ``capacity[s]`` reserved rows: keys (and values) (n_heads, C, d),
    positions (n_heads, C) int32 (-1 on unused rows) and stats {kept, capacity, status, 0}.
    ``values`` must have the dtype and shape of ``keys``.  ``outputs`` may pass back the dict
    of an earlier call with the same shapes to reuse its buffers."""
    torch = _torch()
    keys, dt = _prep_keys(keys)
    H, T, d = keys.shape
    dev = keys.device
    if values is not None:
        if values.dim() == 2:
            values = values.unsqueeze(0)
        if values.dtype != keys.dtype or tuple(values.shape) != (H, T, d) or values.device != dev:
            raise ValueError("values must match keys in dtype, shape and device")
        if values.stride(2) != 1:
            values = values.contiguous()
    cu = _cu(cu_seqlens, T)
    if cu[-1] != T:
        raise ValueError("cu_seqlens[-1] must equal T")
    n_seqs = len(cu) - 1
    ret = _mask(retained, H, T, dev, "retained")
    if ret is None:
        raise ValueError("retained is required")
    cap = np.broadcast_to(np.asarray(capacity, dtype=np.int64), (n_seqs,)).copy()
    C = int(cap.sum())
    if outputs is None:
        out = {
            "keys": torch.empty((H, C, d), dtype=keys.dtype, device=dev),
            "values": torch.empty((H, C, d), dtype=keys.dtype, device=dev) if values is not None else None,
            "pos": torch.empty((H, C), dtype=torch.int32, device=dev) if want_pos else None,
            "stats": torch.empty((H * n_seqs, 4), dtype=torch.int32, device=dev),
        }
    else:
        out = dict(outputs)
        out.setdefault("values", None)
        out.setdefault("pos", None)
    nbytes = workspace_bytes(OP_COMPACT, dt, d, H, cu)
    ws = workspace if workspace is not None and workspace.numel() >= nbytes else \
        torch.empty((nbytes,), dtype=torch.uint8, device=dev)
    vs = (values.stride(0), values.stride(1)) if values is not None else (0, 0)
    rc = lib().twinkv_compact(
        keys.data_ptr(), _ptr(values), dt, d, H, n_seqs, _i64_array(cu), keys.stride(0),
        keys.stride(1), vs[0], vs[1], ret.data_ptr(), _i64_array(cap), out["keys"].data_ptr(),
        _ptr(out["values"]), _ptr(out["pos"]), out["stats"].data_ptr(), ws.data_ptr(), ws.numel(),
        _stream(dev))
    if rc != TWINKV_OK:
        raise TwinKVError("twinkv_compact", rc)
    return {k: v for k, v in out.items() if v is not None}

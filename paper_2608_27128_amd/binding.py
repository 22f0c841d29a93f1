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
NOALLOC_MAX_SEQS = 2048

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
    "twinkv_repair_from_scores_noalloc": (_I, [_VP, _VP, _VP, _I, _I, _PI64, _PI64, _F, _I, _I,
                                               _VP, _VP]),
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
    if keys.dtype == torch.bfloat16:
        dt = TWINKV_BF16
    elif keys.dtype == torch.float32:
        dt = TWINKV_F32
    else:
        raise ValueError(f"unsupported key dtype {keys.dtype}")
    return keys, dt


def _on_gpu(t, name: str):
    """Device check, after the shape and offset checks (which need no GPU)."""
    if not t.is_cuda:
        raise ValueError(f"{name} must be on a GPU")
    if t.dim() == 3 and t.stride(2) != 1:
        t = t.contiguous()
    return t


def _vec2d(x, name: str):
    """A float32 (n_heads, T) or (T,) tensor, before the device check."""
    torch = _torch()
    if x.dim() == 1:
        x = x.unsqueeze(0)
    if x.dim() != 2 or x.dtype != torch.float32:
        raise ValueError(f"{name} must be a float32 (n_heads, T) tensor")
    return x


def _cu(cu_seqlens, T: int):
    """The sequence offsets as int64, checked against the tensors' token count T: the library
    lays every [n_heads][T] buffer out from cu_seqlens, so an offset list that ends anywhere
    but T would make its kernels read or write outside the tensors."""
    if cu_seqlens is None:
        return np.array([0, T], dtype=np.int64)
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    if cu.ndim != 1 or len(cu) < 2:
        raise ValueError("cu_seqlens must list n_seqs + 1 >= 2 offsets")
    if cu[0] != 0 or np.any(np.diff(cu) < 0):
        raise ValueError("cu_seqlens must start at 0 and never decrease")
    if cu[-1] != T:
        raise ValueError(f"cu_seqlens[-1] = {int(cu[-1])} must equal T = {T}")
    return cu


def _check_outputs(out: dict, spec: dict, fn: str) -> dict:
    """Buffers passed back through ``outputs``: each present entry must have the shape, dtype
    and device the call writes (``spec``: name -> (shape, dtype, device, required))."""
    got = dict(out)
    for name, (shape, dtype, dev, required) in spec.items():
        t = got.get(name)
        if t is None:
            if required:
                raise ValueError(f"{fn}: outputs[{name!r}] is required")
            continue
        if tuple(t.shape) != tuple(shape) or t.dtype != dtype or t.device != dev:
            raise ValueError(f"{fn}: outputs[{name!r}] must be {tuple(shape)} {dtype} on {dev}, "
                             f"got {tuple(t.shape)} {t.dtype} on {t.device}")
        if not t.is_contiguous():
            raise ValueError(f"{fn}: outputs[{name!r}] must be contiguous")
    return got


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


def _launch(dev, name: str, *args) -> None:
    """Call the library entry point ``name`` with the tensors' device current: the library
    enqueues on the given stream of the current device and keeps its per-device state there."""
    torch = _torch()
    with torch.cuda.device(dev):
        rc = getattr(lib(), name)(*args)
    if rc != TWINKV_OK:
        raise TwinKVError(name, rc)


def _nbytes(t) -> int:
    return t.numel() * t.element_size()


def _workspace(workspace, nbytes: int, dev):
    """The caller's workspace when it is large enough (a contiguous tensor on the call's
    device; its byte count is what is compared), else a fresh uint8 buffer of nbytes."""
    torch = _torch()
    if workspace is not None:
        if workspace.device != dev or not workspace.is_contiguous():
            raise ValueError(f"workspace must be a contiguous tensor on {dev}")
        if _nbytes(workspace) >= nbytes:
            return workspace
    return torch.empty((nbytes,), dtype=torch.uint8, device=dev)


def nn_scores(keys, retained=None, w: int = 32, cu_seqlens=None, *, want_arg: bool = True,
              workspace=None) -> dict:
    """Best twin of every token: best_all/arg_all over all keys, best_ret/arg_ret (Eq. 4 b_i(S0))
    over the retained set when ``retained`` is given, and a per-problem status."""
    torch = _torch()
    keys, dt = _prep_keys(keys)
    H, T, d = keys.shape
    cu = _cu(cu_seqlens, T)
    keys = _on_gpu(keys, "keys")
    dev = keys.device
    ret = _mask(retained, H, T, dev, "retained")
    out = {
        "best_all": torch.empty((H, T), dtype=torch.float32, device=dev),
        "arg_all": torch.empty((H, T), dtype=torch.int32, device=dev) if want_arg else None,
        "status": torch.empty((H * (len(cu) - 1),), dtype=torch.int32, device=dev),
    }
    if ret is not None:
        out["best_ret"] = torch.empty((H, T), dtype=torch.float32, device=dev)
        out["arg_ret"] = torch.empty((H, T), dtype=torch.int32, device=dev) if want_arg else None
    ws = _workspace(workspace, workspace_bytes(OP_NN_SCORES, dt, d, H, cu), dev)
    _launch(dev, "twinkv_nn_scores",
        keys.data_ptr(), dt, d, H, len(cu) - 1, _i64_array(cu), keys.stride(0), keys.stride(1),
        _ptr(ret), int(w), _ptr(out["best_all"]), _ptr(out["arg_all"]),
        _ptr(out.get("best_ret")), _ptr(out.get("arg_ret")), _ptr(out["status"]),
        ws.data_ptr(), _nbytes(ws), _stream(dev))
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
    cu = _cu(cu_seqlens, T)
    n_seqs = len(cu) - 1
    if level is None:
        raise ValueError("level is required")
    if not 1 <= int(n_levels) <= MAX_LEVELS:
        raise ValueError(f"n_levels must be in [1, {MAX_LEVELS}]")
    keys = _on_gpu(keys, "keys")
    dev = keys.device
    lv = _mask(level, H, T, dev, "level")
    f32, i32 = torch.float32, torch.int32
    spec = {
        "best_lvl": ((n_levels, H, T), f32, dev, True),
        "arg_lvl": ((n_levels, H, T), i32, dev, False),
        "best_all": ((H, T), f32, dev, False),
        "arg_all": ((H, T), i32, dev, False),
        "status": ((H * n_seqs,), i32, dev, True),
    }
    if outputs is None:
        out = {
            "best_lvl": torch.empty((n_levels, H, T), dtype=f32, device=dev),
            "arg_lvl": torch.empty((n_levels, H, T), dtype=i32, device=dev) if want_arg else None,
            "best_all": torch.empty((H, T), dtype=f32, device=dev) if want_all else None,
            "arg_all": torch.empty((H, T), dtype=i32, device=dev) if (want_all and want_arg) else None,
            "status": torch.empty((H * n_seqs,), dtype=i32, device=dev),
        }
    else:
        out = _check_outputs(outputs, spec, "nn_scores_levels")
        want_all = out.get("best_all") is not None or out.get("arg_all") is not None
    ws = _workspace(workspace, levels_workspace_bytes(dt, d, H, cu, n_levels, want_all), dev)
    _launch(dev, "twinkv_nn_scores_levels",
        keys.data_ptr(), dt, d, H, n_seqs, _i64_array(cu), keys.stride(0), keys.stride(1),
        lv.data_ptr(), int(n_levels), int(w), _ptr(out.get("best_all")), _ptr(out.get("arg_all")),
        out["best_lvl"].data_ptr(), _ptr(out.get("arg_lvl")), _ptr(out["status"]),
        ws.data_ptr(), _nbytes(ws), _stream(dev))
    return {k: v for k, v in out.items() if v is not None}


def _budget(budget, n_seqs: int):
    return np.broadcast_to(np.asarray(budget, dtype=np.int64), (n_seqs,)).copy()


def repair(keys, retained, budget, tau: float, w: int = 32, n_sink: int = 4, n_recent: int = 64,
           cu_seqlens=None, *, want_all: bool = True, want_arg: bool = True, out_mask=None,
           workspace=None, outputs: Optional[dict] = None) -> dict:
    """The repair pass of Sec. 3.4: S1 (uint8 mask), stats (|O|, |D|, m, status) per problem,
    and the scores it was computed from (best_ret = b; best_all/arg_all when want_all).

    ``outputs`` may pass back the dict of an earlier call with the same shapes to reuse its
    buffers (the entries it holds decide what is computed); ``out_mask`` may be ``retained``
    itself for an in-place update."""
    torch = _torch()
    keys, dt = _prep_keys(keys)
    H, T, d = keys.shape
    cu = _cu(cu_seqlens, T)
    n_seqs = len(cu) - 1
    if retained is None:
        raise ValueError("retained is required")
    bud = _budget(budget, n_seqs)
    keys = _on_gpu(keys, "keys")
    dev = keys.device
    ret = _mask(retained, H, T, dev, "retained")
    f32, i32 = torch.float32, torch.int32
    if outputs is None:
        out = {
            "s1": torch.empty((H, T), dtype=torch.uint8, device=dev),
            "stats": torch.empty((H * n_seqs, 4), dtype=i32, device=dev),
            "best_ret": torch.empty((H, T), dtype=f32, device=dev),
            "arg_ret": torch.empty((H, T), dtype=i32, device=dev) if want_arg else None,
            "best_all": torch.empty((H, T), dtype=f32, device=dev) if want_all else None,
            "arg_all": torch.empty((H, T), dtype=i32, device=dev) if (want_all and want_arg) else None,
        }
    else:
        spec = {
            "s1": ((H, T), torch.uint8, dev, out_mask is None),
            "stats": ((H * n_seqs, 4), i32, dev, True),
            "best_ret": ((H, T), f32, dev, False),
            "arg_ret": ((H, T), i32, dev, False),
            "best_all": ((H, T), f32, dev, False),
            "arg_all": ((H, T), i32, dev, False),
        }
        out = _check_outputs(outputs, spec, "repair")
    if out_mask is not None:
        m = _mask(out_mask, H, T, dev, "out_mask")
        if m.data_ptr() != out_mask.data_ptr():
            raise ValueError("out_mask must be a contiguous uint8 (n_heads, T) tensor")
        out["s1"] = out_mask
    ws = _workspace(workspace, workspace_bytes(OP_REPAIR, dt, d, H, cu), dev)
    _launch(dev, "twinkv_repair",
        keys.data_ptr(), dt, d, H, n_seqs, _i64_array(cu), keys.stride(0), keys.stride(1),
        ret.data_ptr(), out["s1"].data_ptr(), _i64_array(bud), float(tau), int(w), int(n_sink),
        int(n_recent), out["stats"].data_ptr(), _ptr(out.get("best_all")), _ptr(out.get("arg_all")),
        _ptr(out.get("best_ret")), _ptr(out.get("arg_ret")), ws.data_ptr(), _nbytes(ws), _stream(dev))
    return {k: v for k, v in out.items() if v is not None}


def repair_from_scores(b, retained, budget, tau: float, n_sink: int = 4, n_recent: int = 64,
                       cu_seqlens=None, *, out_mask=None) -> dict:
    """Classification, ranking and swap of Sec. 3.4 from given scores b (n_heads, T) float32."""
    torch = _torch()
    b = _vec2d(b, "b")
    H, T = b.shape
    cu = _cu(cu_seqlens, T)
    n_seqs = len(cu) - 1
    if retained is None:
        raise ValueError("retained is required")
    bud = _budget(budget, n_seqs)
    b = _on_gpu(b, "b").contiguous()
    dev = b.device
    ret = _mask(retained, H, T, dev, "retained")
    if out_mask is not None:
        s1 = _mask(out_mask, H, T, dev, "out_mask")
        if s1.data_ptr() != out_mask.data_ptr():
            raise ValueError("out_mask must be a contiguous uint8 (n_heads, T) tensor")
    else:
        s1 = torch.empty((H, T), dtype=torch.uint8, device=dev)
    stats = torch.empty((H * n_seqs, 4), dtype=torch.int32, device=dev)
    ws = _workspace(None, workspace_bytes(OP_REPAIR_FROM_SCORES, 0, 64, H, cu), dev)
    _launch(dev, "twinkv_repair_from_scores",
        b.data_ptr(), ret.data_ptr(), s1.data_ptr(), H, n_seqs, _i64_array(cu), _i64_array(bud),
        float(tau), int(n_sink), int(n_recent), stats.data_ptr(), ws.data_ptr(), _nbytes(ws),
        _stream(dev))
    return {"s1": s1, "stats": stats}


def repair_from_scores_noalloc(b, retained, budget, tau: float, n_sink: int = 4,
                               n_recent: int = 64, cu_seqlens=None, *, outputs: dict) -> dict:
    """repair_from_scores through the entry point that allocates nothing: the caller passes
    the output buffers (``outputs`` with "s1" uint8 (n_heads, T) and "stats" int32
    (n_heads * n_seqs, 4)), and the library's static scratch holds the sequence table (at
    most NOALLOC_MAX_SEQS sequences).  Calls overlapping on one GPU race."""
    torch = _torch()
    b = _vec2d(b, "b")
    H, T = b.shape
    cu = _cu(cu_seqlens, T)
    n_seqs = len(cu) - 1
    if retained is None:
        raise ValueError("retained is required")
    bud = _budget(budget, n_seqs)
    b = _on_gpu(b, "b")
    if not b.is_contiguous():
        raise ValueError("b must be contiguous (the call may not allocate a copy)")
    dev = b.device
    if retained.dim() == 1:
        retained = retained.unsqueeze(0)
    if (tuple(retained.shape) != (H, T) or retained.dtype != torch.uint8 or retained.device != dev
            or not retained.is_contiguous()):
        raise ValueError(f"retained must be a contiguous uint8 ({H}, {T}) tensor on {dev}")
    spec = {"s1": ((H, T), torch.uint8, dev, True), "stats": ((H * n_seqs, 4), torch.int32, dev, True)}
    out = _check_outputs(outputs, spec, "repair_from_scores_noalloc")
    _launch(dev, "twinkv_repair_from_scores_noalloc",
        b.data_ptr(), retained.data_ptr(), out["s1"].data_ptr(), H, n_seqs, _i64_array(cu),
        _i64_array(bud), float(tau), int(n_sink), int(n_recent), out["stats"].data_ptr(),
        _stream(dev))
    return out


def twin_counts(keys, tau: float, w: int = 32, cu_seqlens=None, *, workspace=None) -> dict:
    """Eq. 2 twin counts r_i (int32, (n_heads, T)) and a per-problem status."""
    torch = _torch()
    keys, dt = _prep_keys(keys)
    H, T, d = keys.shape
    cu = _cu(cu_seqlens, T)
    keys = _on_gpu(keys, "keys")
    dev = keys.device
    counts = torch.empty((H, T), dtype=torch.int32, device=dev)
    status = torch.empty((H * (len(cu) - 1),), dtype=torch.int32, device=dev)
    ws = _workspace(workspace, workspace_bytes(OP_TWIN_COUNTS, dt, d, H, cu), dev)
    _launch(dev, "twinkv_twin_counts",
        keys.data_ptr(), dt, d, H, len(cu) - 1, _i64_array(cu), keys.stride(0), keys.stride(1),
        float(tau), int(w), counts.data_ptr(), status.data_ptr(), ws.data_ptr(), _nbytes(ws),
        _stream(dev))
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
    cu = _cu(cu_seqlens, T)
    n_seqs = len(cu) - 1
    bud = _budget(budget, n_seqs)
    keys = _on_gpu(keys, "keys")
    dev = keys.device
    if outputs is None:
        out = {
            "retained": torch.empty((H, T), dtype=torch.uint8, device=dev),
            "counts": torch.empty((H, T), dtype=torch.int32, device=dev),
            "scores": torch.empty((H, T), dtype=torch.float32, device=dev) if want_scores else None,
            "stats": torch.empty((H * n_seqs, 4), dtype=torch.int32, device=dev),
        }
    else:
        spec = {
            "retained": ((H, T), torch.uint8, dev, True),
            "counts": ((H, T), torch.int32, dev, True),
            "scores": ((H, T), torch.float32, dev, False),
            "stats": ((H * n_seqs, 4), torch.int32, dev, True),
        }
        out = _check_outputs(outputs, spec, "score_evict")
        out.setdefault("scores", None)
    ws = _workspace(workspace, workspace_bytes(OP_SCORE_EVICT, dt, d, H, cu), dev)
    _launch(dev, "twinkv_score_evict",
        keys.data_ptr(), dt, d, H, n_seqs, _i64_array(cu), keys.stride(0), keys.stride(1),
        _i64_array(bud), float(tau), int(w), int(n_sink), int(n_recent),
        out["retained"].data_ptr(), out["counts"].data_ptr(), _ptr(out["scores"]),
        out["stats"].data_ptr(), ws.data_ptr(), _nbytes(ws), _stream(dev))
    return {k: v for k, v in out.items() if v is not None}


def select_topk(scores, budget, n_sink: int = 4, n_recent: int = 64, cu_seqlens=None, *,
                workspace=None, outputs: Optional[dict] = None) -> dict:
    """A score-based policy's retained set (Sec. 3.1 / 3.2): per problem the ``budget[s]``
    positions first in the order protected, higher score, lower position (NaN last).
    scores: float32 (n_heads, T) on the GPU.  Returns retained uint8 (n_heads, T) and
    stats int32 (n_heads * n_seqs, 4) = {kept, NaN scores, 0, 0}."""
    torch = _torch()
    scores = _vec2d(scores, "scores")
    H, T = scores.shape
    cu = _cu(cu_seqlens, T)
    n_seqs = len(cu) - 1
    bud = _budget(budget, n_seqs)
    scores = _on_gpu(scores, "scores").contiguous()
    dev = scores.device
    if outputs is None:
        out = {
            "retained": torch.empty((H, T), dtype=torch.uint8, device=dev),
            "stats": torch.empty((H * n_seqs, 4), dtype=torch.int32, device=dev),
        }
    else:
        spec = {"retained": ((H, T), torch.uint8, dev, True),
                "stats": ((H * n_seqs, 4), torch.int32, dev, True)}
        out = _check_outputs(outputs, spec, "select_topk")
    ws = _workspace(workspace, workspace_bytes(OP_REPAIR_FROM_SCORES, 0, 64, H, cu), dev)
    _launch(dev, "twinkv_select_topk",
        scores.data_ptr(), H, n_seqs, _i64_array(cu), _i64_array(bud), int(n_sink),
        int(n_recent), out["retained"].data_ptr(), _ptr(out["stats"]), ws.data_ptr(),
        _nbytes(ws), _stream(dev))
    return out


def prevalence(best_all, taus, cu_seqlens=None) -> "torch.Tensor":
    """Tokens with at least one twin (best_all > tau) per problem and threshold:
    int32 (n_heads * n_seqs, len(taus))."""
    torch = _torch()
    best_all = _vec2d(best_all, "best_all")
    H, T = best_all.shape
    cu = _cu(cu_seqlens, T)
    n_seqs = len(cu) - 1
    tv = np.ascontiguousarray(np.asarray(taus, dtype=np.float32).reshape(-1))
    if not 1 <= len(tv) <= MAX_TAUS:
        raise ValueError(f"between 1 and {MAX_TAUS} thresholds")
    best_all = _on_gpu(best_all, "best_all").contiguous()
    dev = best_all.device
    out = torch.empty((H * n_seqs, len(tv)), dtype=torch.int32, device=dev)
    ws = _workspace(None, workspace_bytes(OP_REPAIR_FROM_SCORES, 0, 64, H, cu), dev)
    _launch(dev, "twinkv_prevalence",
        best_all.data_ptr(), H, n_seqs, _i64_array(cu),
        tv.ctypes.data_as(ctypes.POINTER(ctypes.c_float)), len(tv), out.data_ptr(),
        ws.data_ptr(), _nbytes(ws), _stream(dev))
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
    if values is not None:
        if values.dim() == 2:
            values = values.unsqueeze(0)
        if values.dtype != keys.dtype or tuple(values.shape) != (H, T, d):
            raise ValueError("values must match keys in dtype and shape")
    cu = _cu(cu_seqlens, T)
    n_seqs = len(cu) - 1
    if retained is None:
        raise ValueError("retained is required")
    cap = _budget(capacity, n_seqs)
    C = int(cap.sum())
    keys = _on_gpu(keys, "keys")
    dev = keys.device
    if values is not None:
        values = _on_gpu(values, "values")
        if values.device != dev:
            raise ValueError("values must be on the keys' device")
    ret = _mask(retained, H, T, dev, "retained")
    if outputs is None:
        out = {
            "keys": torch.empty((H, C, d), dtype=keys.dtype, device=dev),
            "values": torch.empty((H, C, d), dtype=keys.dtype, device=dev) if values is not None else None,
            "pos": torch.empty((H, C), dtype=torch.int32, device=dev) if want_pos else None,
            "stats": torch.empty((H * n_seqs, 4), dtype=torch.int32, device=dev),
        }
    else:
        spec = {
            "keys": ((H, C, d), keys.dtype, dev, True),
            "values": ((H, C, d), keys.dtype, dev, values is not None),
            "pos": ((H, C), torch.int32, dev, False),
            "stats": ((H * n_seqs, 4), torch.int32, dev, True),
        }
        out = _check_outputs(outputs, spec, "compact")
        out.setdefault("values", None)
        out.setdefault("pos", None)
        if values is None:
            out["values"] = None
    ws = _workspace(workspace, workspace_bytes(OP_COMPACT, dt, d, H, cu), dev)
    vs = (values.stride(0), values.stride(1)) if values is not None else (0, 0)
    _launch(dev, "twinkv_compact",
        keys.data_ptr(), _ptr(values), dt, d, H, n_seqs, _i64_array(cu), keys.stride(0),
        keys.stride(1), vs[0], vs[1], ret.data_ptr(), _i64_array(cap), out["keys"].data_ptr(),
        _ptr(out["values"]), _ptr(out["pos"]), out["stats"].data_ptr(), ws.data_ptr(), _nbytes(ws),
        _stream(dev))
    return {k: v for k, v in out.items() if v is not None}

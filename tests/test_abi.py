"""The C-ABI library loads, exports every symbol include/twinkv.h declares, and rejects bad
arguments on the host before enqueueing any GPU work (no GPU needed: validation is host code
and never reaches a HIP call)."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2608_27128_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "twinkv.h")

E_NULL, E_ARG, E_UNSUP, E_WS, E_CAP = 1, 2, 3, 4, 6
FAKE = 0x100000          # 16-byte aligned stand-in for a device pointer; never dereferenced


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(twinkv_\w+)\s*\(", src)))


def test_exports_every_declared_function():
    names = declared_functions()
    assert len(names) >= 6, names
    L = binding.lib()
    for n in names:
        assert hasattr(L, n), f"{n} declared in twinkv.h but not exported"
    assert set(names) == set(binding.SIGNATURES), "binding signatures out of sync with the header"


def test_version_and_strings():
    assert binding.version() == 100
    for code in range(7):
        assert binding.status_string(code) and "unknown" not in binding.status_string(code)
    assert "unknown" in binding.status_string(99)


def cu_arr(v):
    return (ctypes.c_int64 * len(v))(*v)


def test_workspace_bytes():
    L = binding.lib()
    a = L.twinkv_workspace_bytes(0, 0, 128, 8, 1, cu_arr([0, 1000]))
    b = L.twinkv_workspace_bytes(0, 0, 128, 8, 1, cu_arr([0, 2000]))
    assert 0 < a < b
    f32 = L.twinkv_workspace_bytes(0, 1, 64, 8, 1, cu_arr([0, 1000]))
    bf = L.twinkv_workspace_bytes(0, 0, 64, 8, 1, cu_arr([0, 1000]))
    assert f32 > bf                       # fp32 keys add the hi/lo planes
    rep = L.twinkv_workspace_bytes(1, 0, 64, 8, 1, cu_arr([0, 1000]))
    assert rep > bf                       # repair adds the score buffer
    assert L.twinkv_workspace_bytes(2, 0, 0, 8, 1, cu_arr([0, 1000])) > 0
    assert L.twinkv_workspace_bytes(0, 0, 96, 8, 1, cu_arr([0, 10])) == -E_UNSUP
    assert L.twinkv_workspace_bytes(0, 5, 64, 8, 1, cu_arr([0, 10])) == -E_UNSUP
    assert L.twinkv_workspace_bytes(7, 0, 64, 8, 1, cu_arr([0, 10])) == -E_ARG
    tc = L.twinkv_workspace_bytes(3, 0, 64, 8, 1, cu_arr([0, 1000]))
    se = L.twinkv_workspace_bytes(4, 0, 64, 8, 1, cu_arr([0, 1000]))
    assert tc == bf and se > tc           # the scorer adds the count buffer
    # compaction: the sequence table, the chunk list and one count per (head, chunk)
    c1 = L.twinkv_workspace_bytes(5, 0, 0, 8, 1, cu_arr([0, 2048]))
    c2 = L.twinkv_workspace_bytes(5, 0, 0, 8, 1, cu_arr([0, 2049]))
    c3 = L.twinkv_workspace_bytes(5, 0, 0, 8, 3, cu_arr([0, 0, 0, 0]))
    assert 0 < c1 <= c2 and c3 > 0
    assert L.twinkv_workspace_bytes(5, 0, 0, 8, 1, cu_arr([0, 2048 * 300])) > c1 + 4 * 8 * 290
    assert L.twinkv_workspace_bytes(0, 0, 64, 0, 1, cu_arr([0, 10])) == -E_ARG
    assert L.twinkv_workspace_bytes(0, 0, 64, 8, 2, cu_arr([0, 10, 5])) == -E_ARG
    assert L.twinkv_workspace_bytes(0, 0, 64, 8, 1, cu_arr([3, 10])) == -E_ARG
    assert L.twinkv_workspace_bytes(0, 0, 64, 8, 1, None) == -E_NULL


def nn(keys=FAKE, dtype=0, d=64, H=2, cu=(0, 100), hs=6400, ts=64, ret=None, w=32,
       ba=FAKE, aa=FAKE, br=None, ar=None, st=None, ws=FAKE, wsb=1 << 40):
    L = binding.lib()
    return L.twinkv_nn_scores(keys, dtype, d, H, len(cu) - 1, cu_arr(list(cu)), hs, ts, ret, w,
                              ba, aa, br, ar, st, ws, wsb, None)


def test_nn_scores_validation():
    assert nn(keys=None) == E_NULL
    assert nn(d=96) == E_UNSUP
    assert nn(dtype=3) == E_UNSUP
    assert nn(keys=FAKE + 8) == E_ARG          # misaligned
    assert nn(ts=60) == E_ARG                  # token stride shorter than d
    assert nn(ts=68) == E_ARG                  # token stride not a multiple of 16 bytes
    assert nn(hs=-64) == E_ARG
    assert nn(w=-1) == E_ARG
    assert nn(H=0) == E_ARG
    assert nn(cu=(0, 50, 40)) == E_ARG
    assert nn(cu=(1, 50)) == E_ARG
    assert nn(br=FAKE) == E_ARG                # retained reduction without a retained set
    assert nn(ws=None) == E_WS
    assert nn(wsb=16) == E_WS


def rep(keys=FAKE, dtype=0, d=64, H=2, cu=(0, 100), rin=FAKE, rout=FAKE, budget=(50,), tau=0.9,
        w=32, ns=4, nr=64, stats=FAKE, ws=FAKE, wsb=1 << 40):
    L = binding.lib()
    bud = cu_arr(list(budget)) if budget is not None else None
    return L.twinkv_repair(keys, dtype, d, H, len(cu) - 1, cu_arr(list(cu)), 6400, 64, rin, rout,
                           bud, tau, w, ns, nr, stats, None, None, None, None, ws, wsb, None)


def test_repair_validation():
    assert rep(rin=None) == E_NULL
    assert rep(rout=None) == E_NULL
    assert rep(stats=None) == E_NULL
    assert rep(budget=None) == E_NULL
    assert rep(tau=float("nan")) == E_ARG
    assert rep(tau=float("inf")) == E_ARG
    assert rep(budget=(101,)) == E_ARG          # budget larger than the sequence
    assert rep(budget=(-1,)) == E_ARG
    assert rep(ns=-1) == E_ARG
    assert rep(nr=-2) == E_ARG
    assert rep(d=32) == E_UNSUP
    assert rep(wsb=100) == E_WS


def test_repair_from_scores_validation():
    L = binding.lib()

    def call(b=FAKE, rin=FAKE, rout=FAKE, budget=(5,), tau=0.9, ns=0, nr=0, stats=FAKE, wsb=1 << 30):
        return L.twinkv_repair_from_scores(b, rin, rout, 1, 1, cu_arr([0, 10]), cu_arr(list(budget)),
                                           tau, ns, nr, stats, FAKE, wsb, None)
    assert call(b=None) == E_NULL
    assert call(stats=None) == E_NULL
    assert call(tau=float("nan")) == E_ARG
    assert call(budget=(11,)) == E_ARG
    assert call(wsb=0) == E_WS


def test_repair_from_scores_noalloc_validation():
    """Argument and capacity errors come back before any HIP call (no GPU here): the static
    scratch holds the table of at most 2048 sequences."""
    L = binding.lib()

    def call(b=FAKE, s0=FAKE, s1=FAKE, H=2, cu=(0, 100), bud=(50,), tau=0.9, ns=4, nr=8, st=FAKE):
        n = len(cu) - 1
        return L.twinkv_repair_from_scores_noalloc(b, s0, s1, H, n, cu_arr(list(cu)),
                                                   cu_arr(list(bud)), tau, ns, nr, st, None)
    n = binding.NOALLOC_MAX_SEQS
    assert call(b=None) == E_NULL
    assert call(st=None) == E_NULL
    assert call(bud=(101,)) == E_ARG
    assert call(tau=float("nan")) == E_ARG
    assert call(cu=(0, 100, 90), bud=(1, 1)) == E_ARG
    assert call(cu=tuple(range(n + 2)), bud=(1,) * (n + 1)) == E_CAP
    assert "static scratch" in binding.status_string(E_CAP)


def test_twin_counts_validation():
    L = binding.lib()

    def call(keys=FAKE, d=64, tau=0.85, w=32, counts=FAKE, wsb=1 << 40):
        return L.twinkv_twin_counts(keys, 0, d, 2, 1, cu_arr([0, 100]), 6400, 64, tau, w, counts,
                                    None, FAKE, wsb, None)
    assert call(keys=None) == E_NULL
    assert call(counts=None) == E_NULL
    assert call(tau=float("nan")) == E_ARG
    assert call(w=-1) == E_ARG
    assert call(d=96) == E_UNSUP
    assert call(wsb=64) == E_WS


def test_score_evict_validation():
    L = binding.lib()

    def call(budget=(30,), tau=0.85, ns=4, nr=8, rout=FAKE, stats=FAKE, wsb=1 << 40):
        bud = cu_arr(list(budget)) if budget is not None else None
        return L.twinkv_score_evict(FAKE, 0, 64, 2, 1, cu_arr([0, 100]), 6400, 64, bud, tau, 32, ns, nr,
                                    rout, None, None, stats, FAKE, wsb, None)
    assert call(budget=None) == E_NULL
    assert call(rout=None) == E_NULL
    assert call(stats=None) == E_NULL
    assert call(budget=(-1,)) == E_ARG
    assert call(tau=float("inf")) == E_ARG
    assert call(ns=-1) == E_ARG
    assert call(wsb=64) == E_WS


def test_prevalence_validation():
    L = binding.lib()
    taus = (ctypes.c_float * 40)(*([0.5] * 40))

    def call(best=FAKE, n=3, out=FAKE, wsb=1 << 30):
        return L.twinkv_prevalence(best, 2, 1, cu_arr([0, 100]), taus, n, out, FAKE, wsb, None)
    assert call(best=None) == E_NULL
    assert call(out=None) == E_NULL
    assert call(n=0) == E_ARG
    assert call(n=33) == E_ARG                  # more thresholds than one call takes
    assert call(wsb=0) == E_WS


def test_select_topk_validation():
    L = binding.lib()

    def call(scores=FAKE, budget=(10, 20), ns=4, nr=8, out=FAKE, cu=(0, 100, 150), wsb=1 << 30):
        return L.twinkv_select_topk(scores, 2, len(cu) - 1, cu_arr(list(cu)),
                                    None if budget is None else cu_arr(list(budget)), ns, nr, out,
                                    None, FAKE, wsb, None)
    assert call(scores=None) == E_NULL
    assert call(out=None) == E_NULL
    assert call(budget=None) == E_NULL
    assert call(ns=-1) == E_ARG
    assert call(nr=-2) == E_ARG
    assert call(budget=(10, -1)) == E_ARG
    assert call(budget=(2 ** 31, 5)) == E_ARG       # above the documented range
    assert call(cu=(0, 100, 90)) == E_ARG           # decreasing offsets
    assert call(cu=(5, 100, 150)) == E_ARG          # first offset not 0
    assert call(wsb=0) == E_WS


def test_levels_validation():
    L = binding.lib()
    cu = cu_arr([0, 100])
    w1 = L.twinkv_levels_workspace_bytes(0, 64, 2, 1, cu, 1, 0)
    w3 = L.twinkv_levels_workspace_bytes(0, 64, 2, 1, cu, 3, 0)
    w3a = L.twinkv_levels_workspace_bytes(0, 64, 2, 1, cu, 3, 1)
    assert 0 < w1 < w3 < w3a
    assert L.twinkv_levels_workspace_bytes(0, 64, 2, 1, cu, 0, 0) == -E_ARG
    assert L.twinkv_levels_workspace_bytes(0, 64, 2, 1, cu, 5, 0) == -E_ARG
    assert L.twinkv_levels_workspace_bytes(0, 96, 2, 1, cu, 2, 0) == -E_UNSUP

    def call(keys=FAKE, level=FAKE, nl=3, w=32, bl=FAKE, wsb=1 << 40, ts=64):
        return L.twinkv_nn_scores_levels(keys, 0, 64, 2, 1, cu_arr([0, 100]), 6400, ts, level,
                                          nl, w, None, None, bl, None, None, FAKE, wsb, None)
    assert call(keys=None) == E_NULL
    assert call(level=None) == E_NULL
    assert call(bl=None) == E_NULL
    assert call(nl=0) == E_ARG
    assert call(nl=5) == E_ARG
    assert call(w=-1) == E_ARG
    assert call(ts=60) == E_ARG
    assert call(wsb=64) == E_WS


def test_compact_validation():
    L = binding.lib()

    def call(keys=FAKE, vals=FAKE, dtype=0, d=64, cu=(0, 100), hs=6400, ts=64, vhs=6400, vts=64,
             ret=FAKE, cap=(50,), kout=FAKE, vout=FAKE, pos=None, stats=FAKE, wsb=1 << 40):
        c = cu_arr(list(cap)) if cap is not None else None
        return L.twinkv_compact(keys, vals, dtype, d, 2, len(cu) - 1, cu_arr(list(cu)), hs, ts,
                                vhs, vts, ret, c, kout, vout, pos, stats, FAKE, wsb, None)
    assert call(keys=None) == E_NULL
    assert call(ret=None) == E_NULL
    assert call(cap=None) == E_NULL
    assert call(kout=None) == E_NULL
    assert call(stats=None) == E_NULL
    assert call(vout=None) == E_NULL            # values without values_out
    assert call(vals=None) == E_NULL            # values_out without values
    assert call(d=96) == E_UNSUP
    assert call(dtype=3) == E_UNSUP
    assert call(cap=(101,)) == E_ARG            # more rows than the sequence has tokens
    assert call(cap=(-1,)) == E_ARG
    assert call(ts=63) == E_ARG
    assert call(vts=60) == E_ARG                # value rows not 16-byte aligned
    assert call(kout=FAKE + 8) == E_ARG
    assert call(vout=FAKE + 4) == E_ARG
    assert call(keys=FAKE + 2) == E_ARG
    assert call(cu=(0, 60, 50), cap=(1, 1)) == E_ARG
    assert call(wsb=16) == E_WS


def test_binding_refuses_host_tensors():
    torch = pytest.importorskip("torch")
    with pytest.raises(ValueError):
        binding.nn_scores(torch.zeros((4, 64), dtype=torch.bfloat16))


def _no_library(monkeypatch):
    """Any call that reaches the library fails the test: the checks below must come first."""
    def boom():
        raise AssertionError("the wrapper reached the library")
    monkeypatch.setattr(binding, "lib", boom)


@pytest.mark.parametrize("cu", [(0, 40), (0, 80), (0, 30, 70), (0, 70, 64), (5, 64), (64,)])
def test_binding_checks_cu_seqlens_against_T(monkeypatch, cu):
    """Every wrapper refuses offsets that do not end at the tensors' T (64 tokens here), or
    that decrease or do not start at 0, before it calls the library: the library lays each
    [n_heads][T] buffer out from cu_seqlens."""
    torch = pytest.importorskip("torch")
    _no_library(monkeypatch)
    H, T, d = 2, 64, 64
    keys = torch.zeros((H, T, d), dtype=torch.bfloat16)
    mask = torch.zeros((H, T), dtype=torch.uint8)
    f = torch.zeros((H, T), dtype=torch.float32)
    n_seqs = max(1, len(cu) - 1)
    calls = {
        "nn_scores": lambda: binding.nn_scores(keys, mask, 32, cu),
        "nn_scores_levels": lambda: binding.nn_scores_levels(keys, mask, 1, 32, cu),
        "repair": lambda: binding.repair(keys, mask, [0] * n_seqs, 0.9, 32, 4, 4, cu),
        "repair_from_scores": lambda: binding.repair_from_scores(f, mask, [0] * n_seqs, 0.9, 4, 4, cu),
        "twin_counts": lambda: binding.twin_counts(keys, 0.9, 32, cu),
        "score_evict": lambda: binding.score_evict(keys, [0] * n_seqs, 0.9, 32, 4, 4, cu),
        "select_topk": lambda: binding.select_topk(f, [0] * n_seqs, 4, 4, cu),
        "prevalence": lambda: binding.prevalence(f, [0.9], cu),
        "compact": lambda: binding.compact(keys, mask, [0] * n_seqs, cu_seqlens=cu),
    }
    for name, call in calls.items():
        with pytest.raises(ValueError, match="cu_seqlens"):
            call()


def test_binding_checks_passed_outputs(monkeypatch):
    """Buffers passed back through `outputs` are checked against the shapes the call writes
    (the device check comes first, so on a CPU-only host the call stops there, and the shape
    check itself is exercised directly)."""
    torch = pytest.importorskip("torch")
    _no_library(monkeypatch)
    dev = torch.device("cpu")
    good = {"s1": torch.zeros((2, 8), dtype=torch.uint8), "stats": torch.zeros((2, 4), dtype=torch.int32)}
    spec = {"s1": ((2, 8), torch.uint8, dev, True), "stats": ((2, 4), torch.int32, dev, True),
            "best_ret": ((2, 8), torch.float32, dev, False)}
    assert set(binding._check_outputs(good, spec, "repair")) == {"s1", "stats"}
    with pytest.raises(ValueError, match="s1"):
        binding._check_outputs({**good, "s1": torch.zeros((2, 9), dtype=torch.uint8)}, spec, "repair")
    with pytest.raises(ValueError, match="best_ret"):
        binding._check_outputs({**good, "best_ret": torch.zeros((2, 8), dtype=torch.float64)}, spec, "repair")
    with pytest.raises(ValueError, match="stats"):
        binding._check_outputs({"s1": good["s1"]}, spec, "repair")
    with pytest.raises(ValueError, match="contiguous"):
        binding._check_outputs({**good, "s1": torch.zeros((8, 2), dtype=torch.uint8).t()}, spec, "repair")
    # with valid offsets the wrappers stop at the device check on a host tensor
    keys = torch.zeros((2, 8, 64), dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="GPU"):
        binding.repair(keys, good["s1"], 0, 0.9, 32, 4, 4, (0, 8), outputs=good)


def test_missing_library_raises(monkeypatch):
    """No fallback: without the built library every call fails with an error naming it."""
    monkeypatch.setattr(binding, "_lib", None)
    monkeypatch.setattr(binding, "LIB_PATH", os.path.join(ROOT, "no_such_dir", "libtwinkv.so"))
    with pytest.raises(RuntimeError, match="is missing"):
        binding.lib()
    with pytest.raises(RuntimeError, match="is missing"):
        binding.version()


def test_product_package_never_reaches_the_oracle():
    """The package (kernels, C ABI, binding, input generator, build) neither imports nor
    loads anything under oracle/: the oracle is test infrastructure only."""
    pkg = os.path.join(ROOT, "paper_2608_27128_amd")
    offenders = []
    for dirpath, _, files in os.walk(pkg):
        if "_build" in dirpath or "__pycache__" in dirpath:
            continue
        for f in files:
            if not f.endswith((".py", ".hip", ".cpp", ".h")):
                continue
            text = open(os.path.join(dirpath, f), errors="replace").read()
            if re.search(r"^\s*(import\s+oracle|from\s+oracle\b)|oracle/", text, flags=re.M):
                offenders.append(os.path.relpath(os.path.join(dirpath, f), ROOT))
    assert offenders == []


def test_oracle_imports_nothing_of_the_package():
    """The oracle shares no code with the HIP path: it imports numpy and nothing else."""
    src = os.path.join(ROOT, "oracle")
    for f in os.listdir(src):
        if f.endswith(".py"):
            text = open(os.path.join(src, f)).read()
            mods = re.findall(r"^\s*(?:from\s+(\S+)\s+import|import\s+(\S+))", text, flags=re.M)
            names = {a or b for a, b in mods}
            assert names <= {"numpy", "__future__", ".twinkv_oracle"}, (f, names)

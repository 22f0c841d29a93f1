"""Pins for the CPU oracle: checks against what the paper and the mathematics fix.

Each pin takes the oracle module as an argument and raises AssertionError when
the oracle disagrees with a fact that does not come from the oracle itself:
hand-derived fixtures under tests/golden/ (each cites the passage it follows),
closed forms, invariants the repair rule implies, exact no-op cases, and a
property proved from the definitions (idempotence under a stated condition).
``test_oracle_mutants.py`` runs the whole battery on deliberately broken copies
of the oracle and requires every copy to fail at least one pin.
"""
from __future__ import annotations

import json
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _one_hot_keys(one_hot_of, d):
    K = np.zeros((len(one_hot_of), d), dtype=np.float32)
    K[np.arange(len(one_hot_of)), one_hot_of] = 1.0
    return K


# ----------------------------------------------------------------------------
# Eq. 1 / twin rule / Eq. 4
# ----------------------------------------------------------------------------
def pin_closed_forms(o):
    fx = _load("closed_forms.json")
    K = np.asarray(fx["keys"], dtype=np.float32)
    for case in fx["cases"]:
        r = o.nn_scores(K, "f32", None, case["w"])
        np.testing.assert_allclose(r["best_all"], case["best"], rtol=0, atol=1e-12)
        np.testing.assert_array_equal(r["arg_all"], case["arg"])
        np.testing.assert_allclose(r["second_all"], case["second"], rtol=0, atol=1e-12)


def pin_window_and_sentinel(o):
    fx = _load("window_boundary.json")
    K = _one_hot_keys(fx["one_hot_of"], fx["d"])
    ret = np.asarray(fx["retained"], dtype=np.uint8)
    r = o.nn_scores(K, "f32", ret, fx["w"])
    np.testing.assert_array_equal(r["best_all"], fx["best_all"])
    np.testing.assert_array_equal(r["arg_all"], fx["arg_all"])
    np.testing.assert_array_equal(r["best_ret"], fx["best_ret"])
    np.testing.assert_array_equal(r["arg_ret"], fx["arg_ret"])
    sh = fx["short"]
    r = o.nn_scores(K[: sh["n"]], "f32", np.ones(sh["n"], np.uint8), sh["w"])
    for k in ("best_all", "best_ret"):
        np.testing.assert_array_equal(r[k], sh["best"])
    for k in ("arg_all", "arg_ret"):
        np.testing.assert_array_equal(r[k], sh["arg"])
    iw = fx["inside_window"]
    only = np.zeros(iw["n"], np.uint8)
    only[iw["retained_only"]] = 1
    r = o.nn_scores(K[: iw["n"]], "f32", only, iw["w"], rows=np.array([iw["row"]]))
    assert r["best_ret"][0] == iw["best"] and r["arg_ret"][0] == iw["arg"]


def pin_scale_invariance(o):
    """Eq. 1 depends on directions only: positive per-key rescaling leaves every output unchanged."""
    g = np.random.Generator(np.random.PCG64(7))
    K = g.standard_normal((40, 8))
    K[5] = 2.5 * K[30]                        # an exact scaled twin
    ret = (g.random(40) < 0.5).astype(np.uint8)
    a = o.nn_scores(K.astype(np.float32), "f32", ret, 3)
    scale = 2.0 ** g.integers(-6, 7, size=40)  # powers of two keep the float32 inputs exact
    b = o.nn_scores((K * scale[:, None]).astype(np.float32), "f32", ret, 3)
    for k in ("best_all", "best_ret"):
        np.testing.assert_allclose(a[k], b[k], rtol=0, atol=1e-12)
    assert abs(a["best_all"][5] - 1.0) < 1e-12 and a["arg_all"][5] == 30
    # the same pair seen from the other side: symmetry of Eq. 1
    assert abs(a["best_all"][30] - 1.0) < 1e-12 and a["arg_all"][30] == 5


def pin_bf16_decode(o):
    """Raw bf16 bits decode exactly: 0x3F80 = 1.0, 0xC000 = -2.0, 0x4040 = 3.0."""
    bits = np.array([[0x3F80, 0, 0, 0], [0xC000, 0, 0, 0], [0, 0x4040, 0, 0], [0x4040, 0, 0, 0]],
                    dtype=np.uint16)
    r = o.nn_scores(bits, "bf16", None, 0)
    np.testing.assert_allclose(r["best_all"], [1.0, 0.0, 0.0, 1.0], atol=1e-15)
    np.testing.assert_array_equal(r["arg_all"], [3, 2, 0, 0])


def pin_nonfinite_rejected(o):
    K = np.ones((4, 4), np.float32)
    K[2, 1] = np.nan
    try:
        o.nn_scores(K, "f32", None, 0)
    except ValueError:
        return
    raise AssertionError("non-finite keys were accepted")


# ----------------------------------------------------------------------------
# Sec. 3.4 repair
# ----------------------------------------------------------------------------
def pin_repair_ranked(o):
    fx = _load("repair_ranked.json")
    s0 = np.asarray(fx["s0"], dtype=np.uint8)
    for case in fx["cases"]:
        r = o.repair(np.asarray(case["b"]), s0, fx["tau"], fx["n_sink"], fx["n_recent"])
        np.testing.assert_array_equal(r["orphans_ranked"], case["orphans_ranked"])
        np.testing.assert_array_equal(r["donors_ranked"], case["donors_ranked"])
        assert r["m"] == case["m"], (case["name"], r["m"])
        np.testing.assert_array_equal(r["s1"], case["s1"])


def pin_exemption_diagnostics(o):
    """The selection-cut keys of the hand-ranked cases, and the margins' definitions."""
    fx = _load("repair_ranked.json")
    for case in fx["cases"]:
        b = np.asarray(case["b"])
        dg = o.exemption_diagnostics(b, np.asarray(fx["s0"]), fx["tau"], fx["n_sink"], fx["n_recent"],
                                     second=b - 0.25)
        want_o, want_d = case["orphan_cut"], case["donor_cut"]
        assert (dg["orphan_cut"] is None) == (want_o is None), case["name"]
        assert (dg["donor_cut"] is None) == (want_d is None), case["name"]
        if want_o is not None:
            np.testing.assert_allclose(dg["orphan_cut"], want_o, rtol=0, atol=0)
        if want_d is not None:
            np.testing.assert_allclose(dg["donor_cut"], want_d, rtol=0, atol=0)
        np.testing.assert_allclose(dg["tau_margin"][[5, 7, 13]],
                                   [1.85, 0.0, abs(0.84 - 0.85)], rtol=0, atol=1e-15)
        np.testing.assert_allclose(dg["runner_up_margin"], 0.25, rtol=0, atol=1e-15)


def pin_oscillation(o):
    fx = _load("repair_oscillation.json")
    K = _one_hot_keys(fx["one_hot_of"], fx["d"])
    s = np.asarray(fx["s0"], dtype=np.uint8)
    for step in ("pass1", "pass2"):
        exp = fx[step]
        r = o.repair_problem(K, "f32", s, int(s.sum()), fx["tau"], fx["w"], fx["n_sink"], fx["n_recent"])
        np.testing.assert_array_equal(r["best_ret"], exp["b"])
        np.testing.assert_array_equal(r["orphans_ranked"], exp["orphans_ranked"])
        np.testing.assert_array_equal(r["donors_ranked"], exp["donors_ranked"])
        assert r["m"] == exp["m"]
        np.testing.assert_array_equal(r["s1"], exp["s1"])
        s = r["s1"]
    np.testing.assert_array_equal(s, fx["s0"])


def check_repair_invariants(b, s0, tau, n_sink, n_recent, r):
    """Properties every repair result must have (Sec. 3.4), independent of how it is computed."""
    b = np.asarray(b, dtype=np.float64)
    s0 = np.asarray(s0).astype(bool)
    s1 = np.asarray(r["s1"]).astype(bool)
    n = len(b)
    idx = np.arange(n)
    prot = (idx < n_sink) | (idx >= n - n_recent)
    orphan = ~s0 & (b < tau)
    donor = s0 & ~prot & (b >= tau)
    m = min(int(orphan.sum()), int(donor.sum()))
    assert s1.sum() == s0.sum(), "budget changed"
    admitted, evicted = s1 & ~s0, s0 & ~s1
    assert admitted.sum() == m and evicted.sum() == m, "swap count is not min(|O|,|D|)"
    assert not (admitted & ~orphan).any(), "admitted a non-orphan"
    assert not (evicted & ~donor).any(), "evicted a non-donor"
    assert not (s0 & prot & ~s1).any(), "evicted a protected token"
    # severity: every admitted orphan ranks before every orphan left out (b asc, index asc)
    key_o = lambda i: (b[i], i)
    key_d = lambda i: (-b[i], i)
    out_o = idx[orphan & ~admitted]
    out_d = idx[donor & ~evicted]
    if m and len(out_o):
        assert max(map(key_o, idx[admitted])) < min(map(key_o, out_o)), "orphan severity order"
    if m and len(out_d):
        assert max(map(key_d, idx[evicted])) < min(map(key_d, out_d)), "donor severity order"
    assert r["m"] == m and r["n_orphan"] == int(orphan.sum()) and r["n_donor"] == int(donor.sum())


def pin_repair_invariants(o):
    g = np.random.Generator(np.random.PCG64(11))
    for t in range(300):
        n = int(g.integers(1, 60))
        # quantised scores create many exact ties, including values equal to tau
        b = np.round(g.uniform(-1.0, 1.0, n) * 8) / 8
        b[g.random(n) < 0.1] = -1.0
        s0 = (g.random(n) < g.uniform(0.1, 0.9)).astype(np.uint8)
        tau = float(np.round(g.uniform(-0.5, 1.0) * 8) / 8)
        n_sink, n_recent = int(g.integers(0, 4)), int(g.integers(0, 4))
        r = o.repair(b, s0, tau, n_sink, n_recent)
        check_repair_invariants(b, s0, tau, n_sink, n_recent, r)


def pin_exact_noops(o):
    """tau above every cosine -> no donors; tau below every b (b >= -1) -> no orphans."""
    g = np.random.Generator(np.random.PCG64(3))
    for t in range(20):
        n = int(g.integers(8, 80))
        K = g.standard_normal((n, 8)).astype(np.float32)
        K[n // 2] = K[1]
        s0 = (g.random(n) < 0.5).astype(np.uint8)
        for tau in (1.5, -1.5):
            r = o.repair_problem(K, "f32", s0, int(s0.sum()), tau, 2, 1, 1)
            np.testing.assert_array_equal(r["s1"], s0)
            assert r["m"] == 0
            if tau > 1:
                assert r["n_donor"] == 0
            else:
                assert r["n_orphan"] == 0


def pin_redundancy_consistent_noop(o):
    """The paper's no-op check (Sec. 3.4, Sec. 4.1): when every evicted token has a retained
    twin and no retained token has a retained twin, both sets are empty and S1 = S0."""
    g = np.random.Generator(np.random.PCG64(5))
    for t in range(100):
        n = int(g.integers(6, 48))
        w = int(g.integers(0, 4))
        s0 = (g.random(n) < 0.5).astype(np.uint8)
        s0[0] = 1
        ret = np.flatnonzero(s0)
        d = len(ret) + 1
        K = np.zeros((n, d), np.float32)
        K[ret, np.arange(len(ret))] = 1.0            # retained keys: mutually orthogonal
        ok = True
        for i in np.flatnonzero(s0 == 0):            # evicted: copy of a retained key beyond w
            far = ret[np.abs(ret - i) > w]
            if len(far) == 0:
                ok = False
                break
            K[i] = K[far[g.integers(len(far))]]
        if not ok:
            continue
        for tau in (0.85, 0.9, 1.0):
            r = o.repair_problem(K, "f32", s0, int(s0.sum()), tau, w, 0, 0)
            assert r["n_orphan"] == 0 and r["n_donor"] == 0
            np.testing.assert_array_equal(r["s1"], s0)


def pin_second_pass_condition(o):
    """If |D| <= |O| and no two admitted orphans are twins of each other (sim >= tau beyond w),
    a second pass finds no donors and leaves S1 unchanged.  Proof: a retained non-donor j cannot
    gain an admitted orphan o as a twin, because sim(j, o) >= tau with j in S0 and |j-o| > w
    would have given o a surviving twin; and an admitted orphan's best retained similarity is
    below tau by the condition.  The check runs on random small caches with planted twins."""
    g = np.random.Generator(np.random.PCG64(13))
    hits = 0
    for t in range(150):
        n = int(g.integers(10, 64))
        d = 8
        w = int(g.integers(0, 3))
        K = g.standard_normal((n, d))
        for _ in range(n // 3):
            a, b_ = g.integers(0, n, size=2)
            K[a] = K[b_] + 0.05 * g.standard_normal(d)
        K = K.astype(np.float32)
        s0 = (g.random(n) < 0.5).astype(np.uint8)
        tau = 0.9
        r1 = o.repair_problem(K, "f32", s0, int(s0.sum()), tau, w, 1, 1)
        if not (r1["n_donor"] <= r1["n_orphan"]):
            continue
        adm = np.flatnonzero(r1["s1"].astype(bool) & ~s0.astype(bool))
        Kd = K.astype(np.float64)
        nrm = np.linalg.norm(Kd, axis=1)
        twins = False
        for x in range(len(adm)):
            for y in range(x + 1, len(adm)):
                i, j = adm[x], adm[y]
                if abs(i - j) > w and Kd[i] @ Kd[j] / (nrm[i] * nrm[j]) >= tau:
                    twins = True
        if twins:
            continue
        r2 = o.repair_problem(K, "f32", r1["s1"], int(s0.sum()), tau, w, 1, 1)
        assert r2["n_donor"] == 0, "second pass found donors although the condition holds"
        np.testing.assert_array_equal(r2["s1"], r1["s1"])
        hits += 1
    assert hits >= 20, hits


def pin_budget_checked(o):
    K = np.eye(6, dtype=np.float32)
    s0 = np.array([1, 1, 0, 0, 1, 0], np.uint8)
    try:
        o.repair_problem(K, "f32", s0, 2, 0.9, 0, 0, 0)
    except ValueError:
        return
    raise AssertionError("budget != |S0| was accepted")


# ----------------------------------------------------------------------------
# Eq. 2-3 scorer and the Fig. 1b prevalence
# ----------------------------------------------------------------------------
def pin_twin_counts_golden(o):
    fx = _load("twin_counts.json")
    K = _one_hot_keys(fx["group"], fx["d"])
    for case in fx["cases"]:
        c = o.twin_counts(K, "f32", fx["tau"], case["w"])["counts"]
        np.testing.assert_array_equal(c, case["counts"])
    st = fx["strict"]
    K = np.asarray(st["keys"], dtype=np.float32)
    np.testing.assert_array_equal(o.twin_counts(K, "f32", 0.5, st["w"])["counts"], st["counts_at_0.5"])
    np.testing.assert_array_equal(o.twin_counts(K, "f32", 0.4999, st["w"])["counts"],
                                  st["counts_at_0.4999"])


def pin_twin_counts_band(o):
    """The margin band the count parity tests rely on: counts at tau + margin and at
    tau - margin, window respected, strict comparisons (hand-derived, exact arithmetic)."""
    fx = _load("twin_counts.json")
    st, band = fx["strict"], fx["band"]
    K = np.asarray(st["keys"], dtype=np.float32)
    for case in band["cases"]:
        r = o.twin_counts(K, "f32", case["tau"], st["w"], margin=case["margin"])
        for key in ("counts", "counts_lo", "counts_hi"):
            np.testing.assert_array_equal(r[key], case[key], err_msg=f"{key} at tau {case['tau']}")
    # the band is ordered and collapses to the counts at margin 0+
    rng = np.random.default_rng(13)
    K = rng.standard_normal((60, 8)).astype(np.float32)
    K[30:45] = K[5:20] + np.float32(0.05) * rng.standard_normal((15, 8)).astype(np.float32)
    r = o.twin_counts(K, "f32", 0.8, 3, margin=0.05)
    assert np.all(r["counts_lo"] <= r["counts"]) and np.all(r["counts"] <= r["counts_hi"])
    assert np.any(r["counts_lo"] < r["counts_hi"])
    assert "counts_lo" not in o.twin_counts(K, "f32", 0.8, 3)


def _brute_counts(K, tau, w):
    """Pure-Python Eq. 2 on a tiny input: its own normalisation and dot products."""
    import math
    n = len(K)
    norms = [math.sqrt(math.fsum(float(x) * float(x) for x in k)) for k in K]
    out = []
    for i in range(n):
        c = 0
        for j in range(n):
            if abs(i - j) <= w or norms[i] == 0.0 or norms[j] == 0.0:
                continue
            s = math.fsum(float(a) * float(b) for a, b in zip(K[i], K[j])) / (norms[i] * norms[j])
            assert abs(s - tau) > 1e-9, "brute-force case too close to the threshold"
            c += s > tau
        out.append(c)
    return out


def _brute_best(K, member, w):
    """Pure-Python Eq. 1 maximised over j with |i-j| > w (Sec. 3.2's window) and, when member
    is given, j in that set (Eq. 4): its own norms and dot products, a zero key at similarity
    0 with everything.  Per row: (best, smallest maximising j, best of the other values, the
    similarity of every candidate j), with (-1, -1, -inf, {}) where no j qualifies."""
    import math
    n = len(K)
    norms = [math.sqrt(math.fsum(float(x) * float(x) for x in k)) for k in K]
    out = []
    for i in range(n):
        cand = []
        for j in range(n):
            if abs(i - j) <= w or (member is not None and not member[j]):
                continue
            if norms[i] == 0.0 or norms[j] == 0.0:
                s = 0.0
            else:
                s = math.fsum(float(a) * float(b) for a, b in zip(K[i], K[j])) / (norms[i] * norms[j])
            cand.append((s, j))
        if not cand:
            out.append((-1.0, -1, -math.inf, {}))
            continue
        best = max(s for s, _ in cand)
        arg = min(j for s, j in cand if s == best)
        rest = [s for s, _ in cand if s != best]
        out.append((best, arg, max(rest) if rest else -math.inf, dict((j, s) for s, j in cand)))
    return out


def pin_nn_scores_brute_force(o):
    """Eq. 1 and Eq. 4 against a pure-Python brute force on tiny inputs: random keys with
    exact duplicates (ties go to the smallest position), zero keys, windows from 0 to past
    the sequence, and retained sets from empty to full."""
    rng = np.random.default_rng(21)
    for trial in range(12):
        n, d = int(rng.integers(2, 17)), int(rng.integers(1, 6))
        w = int(rng.choice([0, 1, 2, 3, n]))
        K = rng.standard_normal((n, d)).astype(np.float32)
        for _ in range(int(rng.integers(0, 3))):   # exact duplicates: exact ties
            a, b = rng.choice(n, 2, replace=False)
            K[b] = K[a]
        if trial % 3 == 0:
            K[rng.integers(n)] = 0.0
        member = (rng.random(n) < [0.0, 0.5, 1.0][trial % 3]).astype(np.uint8)
        r = o.nn_scores(K, "f32", member, w)
        for kind, mem in (("all", None), ("ret", member)):
            for i, (best, arg, other, cand) in enumerate(_brute_best(K.tolist(), mem, w)):
                got = int(r["arg_" + kind][i])
                assert abs(r["best_" + kind][i] - best) < 1e-12, (trial, kind, i)
                if best - other > 1e-9:      # exact ties only: the smallest position
                    assert got == arg, (trial, kind, i)
                else:                        # a near-tie: any candidate within 1e-9 of the best
                    assert got in cand and cand[got] >= best - 1e-9, (trial, kind, i)


def pin_twin_counts_brute_force(o):
    rng = np.random.default_rng(11)
    for trial in range(6):
        n, d, w = 14, 4, int(rng.integers(0, 4))
        K = rng.standard_normal((n, d)).astype(np.float32)
        for _ in range(3):                      # a few near-copies, so counts are not all 0
            a, b = rng.choice(n, 2, replace=False)
            K[b] = K[a] + np.float32(0.05) * rng.standard_normal(d).astype(np.float32)
        tau = float(rng.choice([0.0, 0.3, 0.8, 0.95]))
        np.testing.assert_array_equal(o.twin_counts(K, "f32", tau, w)["counts"],
                                      _brute_counts(K.tolist(), tau, w))


def pin_twin_counts_vs_best(o):
    """A token has a twin (r_i >= 1) exactly when its best similarity outside the window
    exceeds tau: the count path and the max path must agree; pairs are counted from both
    sides, so the counts sum to an even number."""
    rng = np.random.default_rng(12)
    K = rng.standard_normal((300, 8)).astype(np.float32)
    src = rng.integers(0, 280, 40)
    K[src + rng.integers(5, 20, 40)] = K[src] + np.float32(0.05) * rng.standard_normal((40, 8)).astype(np.float32)
    for tau in (0.5, 0.9, 0.99):
        for w in (0, 3, 10):
            c = o.twin_counts(K, "f32", tau, w)["counts"]
            b = o.nn_scores(K, "f32", None, w)["best_all"]
            np.testing.assert_array_equal(c >= 1, b > tau)
            assert int(c.sum()) % 2 == 0


def pin_scores_eq3(o):
    c = np.array([0, 1, 5, 2])
    np.testing.assert_allclose(o.redundancy_scores(c, 8), [0.0, -0.125, -0.625, -0.25], rtol=0, atol=0)


def pin_evict_golden(o):
    fx = _load("evict_ranked.json")
    for case in fx["cases"]:
        got = o.evict_by_score(np.asarray(fx["counts"]), case["budget"], fx["n_sink"], fx["n_recent"])
        np.testing.assert_array_equal(got, case["retained"])


def pin_evict_invariants(o):
    """Budget exactly met, protected regions kept, every kept token scores at least as high
    as every evicted one, and at the cut the later positions are the kept ones."""
    rng = np.random.default_rng(13)
    for trial in range(200):
        n = int(rng.integers(1, 40))
        counts = rng.integers(0, 4, n)          # many exact ties
        n_sink, n_recent = int(rng.integers(0, 4)), int(rng.integers(0, 4))
        budget = int(rng.integers(0, n + 3))
        keep = o.evict_by_score(counts, budget, n_sink, n_recent).astype(bool)
        assert keep.sum() == min(budget, n)
        idx = np.arange(n)
        prot = (idx < n_sink) | (idx >= n - n_recent)
        if budget >= prot.sum():
            assert keep[prot].all()
        free = ~prot
        kept, ev = keep & free, ~keep & free
        if kept.any() and ev.any():
            assert counts[kept].max() <= counts[ev].min()
            cut = counts[kept].max()
            if (ev & (counts == cut)).any():
                assert idx[kept & (counts == cut)].min() > idx[ev & (counts == cut)].max()
        if budget < prot.sum():
            assert not keep[free].any()


def pin_prevalence_golden(o):
    fx = _load("prevalence.json")
    np.testing.assert_array_equal(o.prevalence(np.asarray(fx["best"]), fx["taus"]), fx["counts"])


# ----------------------------------------------------------------------------
# Sec. 3.1 / 3.2: a score-based policy's retained set (reading R22)
# ----------------------------------------------------------------------------
def pin_select_golden(o):
    fx = _load("select_topk.json")
    scores = np.array([float(x) for x in fx["scores"]])
    for case in fx["cases"]:
        got = o.select_topk(scores, case["budget"], fx["n_sink"], fx["n_recent"])
        np.testing.assert_array_equal(got, case["retained"])


def _ahead(i, j, sc, prot):
    """True when position j precedes position i in the retention order, decided pairwise:
    protected before unprotected; inside the protected regions, by position; otherwise a
    number before NaN, then the higher score, then the lower position."""
    if prot[j] != prot[i]:
        return bool(prot[j])
    if prot[j]:
        return j < i
    nj, ni = np.isnan(sc[j]), np.isnan(sc[i])
    if nj != ni:
        return bool(ni)
    if not nj and sc[j] != sc[i]:
        return bool(sc[j] > sc[i])
    return j < i


def pin_select_brute_force(o):
    """Position i is kept exactly when fewer than `budget` positions precede it (pairwise
    comparison, no sorting), on tiny problems with many ties, signed zeros, infinities and
    NaN; the protected regions overlap or cover everything in some draws."""
    rng = np.random.default_rng(23)
    pool = np.array([0.0, -0.0, 0.5, -0.5, 1.0, np.inf, -np.inf, np.nan])
    for trial in range(300):
        n = int(rng.integers(0, 14))
        sc = pool[rng.integers(0, len(pool), n)]
        n_sink, n_recent = int(rng.integers(0, 4)), int(rng.integers(0, 4))
        budget = int(rng.integers(0, n + 3))
        idx = np.arange(n)
        prot = (idx < n_sink) | (idx >= n - n_recent)
        want = np.array([sum(_ahead(i, j, sc, prot) for j in range(n) if j != i) < budget
                         for i in range(n)], dtype=np.uint8)
        np.testing.assert_array_equal(o.select_topk(sc, budget, n_sink, n_recent), want)


def pin_select_invariants(o):
    """|S| = min(K, n); the protected regions are kept when K >= |P| and only they (lowest
    positions first) otherwise; every kept score is at least every dropped one; NaN only
    after every number; at the cut the kept positions are the lower ones."""
    rng = np.random.default_rng(29)
    for trial in range(200):
        n = int(rng.integers(1, 60))
        sc = np.round(rng.standard_normal(n), 1)          # many exact ties
        sc[rng.random(n) < 0.1] = np.nan
        n_sink, n_recent = int(rng.integers(0, 5)), int(rng.integers(0, 5))
        budget = int(rng.integers(0, n + 3))
        keep = o.select_topk(sc, budget, n_sink, n_recent).astype(bool)
        assert keep.sum() == min(budget, n)
        idx = np.arange(n)
        prot = (idx < n_sink) | (idx >= n - n_recent)
        if budget >= prot.sum():
            assert keep[prot].all()
        else:
            assert np.array_equal(idx[keep], idx[prot][:budget])
            continue
        free = ~prot
        kept, ev = keep & free, ~keep & free
        if (kept & np.isnan(sc)).any():
            assert not (ev & ~np.isnan(sc)).any()
        kn, en = kept & ~np.isnan(sc), ev & ~np.isnan(sc)
        if kn.any() and en.any():
            assert sc[kn].min() >= sc[en].max()
            cut = sc[kn].min()
            if (en & (sc == cut)).any():
                assert idx[kn & (sc == cut)].max() < idx[en & (sc == cut)].min()


# ----------------------------------------------------------------------------
# Sec. 3.1: the compacted cache
# ----------------------------------------------------------------------------
def pin_compact_golden(o):
    fx = _load("compact.json")
    H, T = len(fx["retained"]), fx["cu_seqlens"][-1]
    t = np.arange(T)
    keys = np.stack([np.stack([10 * h + t, -(10 * h + t)], axis=1) for h in range(H)]).astype(np.int32)
    vals = np.stack([np.stack([100 + 10 * h + t, 200 + 10 * h + t], axis=1)
                     for h in range(H)]).astype(np.int32)
    r = o.compact(keys, vals, np.asarray(fx["retained"], dtype=np.uint8), fx["cu_seqlens"],
                  fx["capacity"])
    np.testing.assert_array_equal(r["keys"], fx["keys_out"])
    np.testing.assert_array_equal(r["values"], fx["values_out"])
    np.testing.assert_array_equal(r["pos"], fx["pos"])
    np.testing.assert_array_equal(r["stats"], fx["stats"])


def pin_compact_invariants(o):
    """The rows of a problem are exactly its kept rows, each once, in position order; the
    rest is zero with position -1; bytes are copied unchanged (NaN payloads included)."""
    rng = np.random.default_rng(17)
    for trial in range(100):
        n = int(rng.integers(0, 30))
        d = int(rng.integers(1, 5))
        bits = rng.integers(0, 2 ** 16, (n, d)).astype(np.uint16)   # arbitrary bf16 patterns
        vbits = rng.integers(0, 2 ** 16, (n, d)).astype(np.uint16)
        keep = (rng.random(n) < rng.random()).astype(np.uint8)
        cap = int(rng.integers(0, n + 3))
        r = o.compact_problem(bits, vbits, keep, cap)
        k = int(keep.sum())
        assert r["stats"][0] == k and r["stats"][1] == cap
        if k > cap:
            assert r["stats"][2] == 1
            assert not r["keys"].any() and not r["values"].any() and np.all(r["pos"] == -1)
            continue
        assert r["stats"][2] == 0
        pos = r["pos"][:k]
        assert np.all(np.diff(pos) > 0) and set(pos.tolist()) == set(np.flatnonzero(keep).tolist())
        for row, p in enumerate(pos):
            assert np.array_equal(r["keys"][row], bits[p]) and np.array_equal(r["values"][row], vbits[p])
        assert not r["keys"][k:].any() and not r["values"][k:].any() and np.all(r["pos"][k:] == -1)


ALL_PINS = [
    pin_closed_forms, pin_window_and_sentinel, pin_scale_invariance, pin_bf16_decode,
    pin_nonfinite_rejected, pin_repair_ranked, pin_oscillation, pin_repair_invariants,
    pin_exact_noops, pin_redundancy_consistent_noop, pin_second_pass_condition,
    pin_budget_checked, pin_nn_scores_brute_force,
    pin_twin_counts_golden, pin_twin_counts_band, pin_twin_counts_brute_force, pin_twin_counts_vs_best,
    pin_scores_eq3, pin_evict_golden, pin_evict_invariants, pin_prevalence_golden,
    pin_compact_golden, pin_compact_invariants, pin_exemption_diagnostics,
    pin_select_golden, pin_select_brute_force, pin_select_invariants,
]

"""The GPU parity protocol (tests/gpu_util.py) on the CPU: scores perturbed within the
similarity tolerance, repaired by the oracle's own logic, must pass check_repair, and a
retained set with a planted mistake (a swap far from every tie, a wrong count, a donor left
in place) must fail it.  No GPU is involved: the "GPU" side here is simulated."""
import numpy as np
import pytest

import oracle
from gpu_util import check_every_row, check_repair, check_scores


def _problem(seed, n=400, d=16, tau=0.9, w=4):
    rng = np.random.default_rng(seed)
    K = rng.standard_normal((n, d)).astype(np.float32)
    src = rng.integers(0, n - 40, n // 4)
    K[src + rng.integers(w + 1, 30, len(src))] = K[src] + np.float32(0.2) * rng.standard_normal((len(src), d)).astype(np.float32)
    s0 = np.zeros(n, np.uint8)
    s0[rng.choice(n, n // 2, replace=False)] = 1
    budget = int(s0.sum())
    orc = oracle.repair_problem(K, "f32", s0, budget, tau, w, 2, 3)
    return K, s0, orc, tau, w


def _simulate(orc, s0, tau, noise, seed):
    rng = np.random.default_rng(seed)
    b = orc["best_ret"] + noise * rng.uniform(-1, 1, len(s0))
    r = oracle.repair(b, s0, tau, 2, 3)
    stats = np.array([r["n_orphan"], r["n_donor"], r["m"], 0])
    return b, r["s1"], stats


@pytest.mark.parametrize("seed", range(6))
def test_perturbed_scores_pass(seed):
    K, s0, orc, tau, w = _problem(seed)
    b, s1, stats = _simulate(orc, s0, tau, 3e-5, seed)
    res = check_repair(s1, stats, b, orc, s0, tau, 2, 3)
    assert res["m"] == stats[2]


def test_flags_flipped_near_tau_pass():
    """A score placed exactly at tau on the oracle side and just below on the GPU side flips
    one flag; the set may then differ, within the allowance."""
    K, s0, orc, tau, w = _problem(3)
    b = orc["best_ret"].copy()
    evicted = np.flatnonzero(~s0.astype(bool) & (b >= tau))
    if not len(evicted):
        pytest.skip("no evicted token with a twin in this draw")
    i = evicted[0]
    orc = dict(orc)
    orc["best_ret"] = orc["best_ret"].copy()
    orc["best_ret"][i] = tau + 2e-4          # the oracle's token sits just above tau ...
    r_o = oracle.repair(orc["best_ret"], s0, tau, 2, 3)
    orc.update(s1=r_o["s1"], orphan=r_o["orphan"], donor=r_o["donor"])
    b[i] = tau - 2e-4                         # ... the GPU's just below: it becomes an orphan
    r = oracle.repair(b, s0, tau, 2, 3)
    res = check_repair(r["s1"], np.array([r["n_orphan"], r["n_donor"], r["m"], 0]), b, orc, s0, tau, 2, 3)
    assert res["flag_diff"] == 1


def test_planted_far_swap_fails():
    K, s0, orc, tau, w = _problem(1)
    b, s1, stats = _simulate(orc, s0, tau, 3e-5, 1)
    s1 = s1.copy()
    adm = np.flatnonzero(s1.astype(bool) & ~s0.astype(bool))
    other = np.flatnonzero(~s1.astype(bool) & ~s0.astype(bool) & (orc["best_ret"] < tau - 0.05))
    assert len(adm) and len(other)
    # admit a different orphan than the most severe ones: far from the cut, same counts
    far = other[np.argmax(orc["best_ret"][other])]
    s1[adm[0]] = 0
    s1[far] = 1
    with pytest.raises(AssertionError):
        check_repair(s1, stats, b, orc, s0, tau, 2, 3)


def test_planted_wrong_stats_fail():
    K, s0, orc, tau, w = _problem(2)
    b, s1, stats = _simulate(orc, s0, tau, 3e-5, 2)
    bad = stats.copy()
    bad[2] += 1
    with pytest.raises(AssertionError):
        check_repair(s1, bad, b, orc, s0, tau, 2, 3)


def test_planted_unswapped_donor_fails():
    K, s0, orc, tau, w = _problem(4)
    b, s1, stats = _simulate(orc, s0, tau, 3e-5, 4)
    s1 = s1.copy()
    ev = np.flatnonzero(s0.astype(bool) & ~s1.astype(bool))
    adm = np.flatnonzero(s1.astype(bool) & ~s0.astype(bool))
    assert len(ev) and len(adm)
    s1[ev[0]] = 1
    s1[adm[0]] = 0
    with pytest.raises(AssertionError):
        check_repair(s1, stats, b, orc, s0, tau, 2, 3)


def test_flag_flip_far_from_tau_fails():
    K, s0, orc, tau, w = _problem(5)
    b = orc["best_ret"].copy()
    far = np.flatnonzero(~s0.astype(bool) & (b < tau - 0.1))
    b[far[0]] = tau + 0.01                    # an orphan the GPU would wrongly see as covered
    r = oracle.repair(b, s0, tau, 2, 3)
    with pytest.raises(AssertionError):
        check_repair(r["s1"], np.array([r["n_orphan"], r["n_donor"], r["m"], 0]), b, orc, s0, tau, 2, 3)


def test_value_bound_enforced():
    """Scores 2e-4 off pass the 1e-3 tolerance but not the 1e-4 bound the library states."""
    K, s0, orc, tau, w = _problem(0, n=120)
    rows = np.arange(120)
    full = oracle.nn_scores(K, "f32", s0, w)
    g = {k: full[k].copy() for k in ("best_all", "arg_all", "best_ret", "arg_ret")}
    check_scores(g, full, rows, K, "f32", s0, w)
    v = g["best_all"] >= 0
    g["best_all"] = np.where(v, g["best_all"] + 2e-4, g["best_all"])
    with pytest.raises(AssertionError, match="stated bound"):
        check_scores(g, full, rows, K, "f32", s0, w)


def test_rank_error_beyond_tolerance_fails():
    """A GPU score off by 5e-3 at the orphan cut reorders the selection in a way that is
    consistent with the GPU's own b (the replay passes) but not within tolerance of the
    exact cut: the per-token cut rule must catch it, while an error of 3e-5 passes."""
    n = 40
    s0 = np.zeros(n, np.uint8)
    s0[:20] = 1
    b_o = np.full(n, 0.95)                   # retained tokens 5..19 are donors (sinks 0, 1)
    b_o[20:] = 0.5 + 0.01 * np.arange(20)    # 20 orphans, 0.01 apart ...
    b_o[25], b_o[26] = 0.5504, 0.5506        # ... but the 6th and 7th only 2e-4 apart
    b_o[2:14] = 0.5                          # only 6 donors (14..19): m = 6 cuts the orphans
    r_o = oracle.repair(b_o, s0, 0.9, 2, 0)
    assert r_o["m"] == 6                     # orphans 20..25 admitted, the cut between 25 and 26
    orc = {"best_ret": b_o, "s1": r_o["s1"], "orphan": r_o["orphan"], "donor": r_o["donor"]}

    def run(b):
        r = oracle.repair(b, s0, 0.9, 2, 0)
        return check_repair(r["s1"], np.array([r["n_orphan"], r["n_donor"], r["m"], 0]), b, orc, s0, 0.9, 2, 0)

    b = b_o.copy()
    b[26] -= 3e-4                             # within tolerance: 26 now precedes 25 at the cut
    assert run(b)["cut_diff"] == 2
    b = b_o.copy()
    b[24] += 0.015                            # 5e-3 past orphan 25: a rank error beyond tolerance
    with pytest.raises(AssertionError, match="cut"):
        run(b)


def _every_row_case():
    """Two ragged heads (an empty sequence, one shorter than the window) with the oracle's own
    best twins in the [n_heads][T] layout check_every_row reads."""
    rng = np.random.default_rng(5)
    cu = np.array([0, 300, 300, 330, 336], np.int64)
    H, T, d, w = 2, int(cu[-1]), 8, 4
    K = rng.standard_normal((H, T, d)).astype(np.float32)
    K[0, 40] = K[0, 10]                                  # an exact tie
    ret = (rng.random((H, T)) < 0.5).astype(np.uint8)
    ret[1, 330:336] = 0                                  # a sequence with an empty S0
    g = {k: np.full((H, T), -1.0 if k.startswith("best") else -1) for k in
         ("best_all", "arg_all", "best_ret", "arg_ret")}
    for h in range(H):
        for s in range(len(cu) - 1):
            a, e = int(cu[s]), int(cu[s + 1])
            if e > a:
                r = oracle.nn_scores(K[h, a:e], "f32", ret[h, a:e], w)
                for k in g:
                    g[k][h, a:e] = r[k]
    return K, ret, cu, w, g


def test_every_row_check_accepts_the_oracle():
    K, ret, cu, w, g = _every_row_case()
    st = check_every_row(K, "f32", ret, cu, w, g)
    assert st["rows_with_candidate"] > 1000 and st["rows_without"] > 0


@pytest.mark.parametrize("mistake", ["moved", "in_window", "sentinel_with_candidates",
                                     "candidate_without_members", "non_member", "value_off",
                                     "asymmetric"])
def test_every_row_check_rejects_planted_mistakes(mistake):
    K, ret, cu, w, g = _every_row_case()
    g = {k: v.copy() for k, v in g.items()}
    i = int(np.nonzero(g["arg_all"][0, :300] >= 0)[0][7])
    if mistake == "moved":                       # another position, far from a tie
        g["arg_all"][0, i] = (g["arg_all"][0, i] + 97) % 300
    elif mistake == "in_window":
        g["arg_all"][0, i] = i + 1
    elif mistake == "sentinel_with_candidates":
        g["arg_ret"][0, i], g["best_ret"][0, i] = -1, -1.0
    elif mistake == "candidate_without_members":     # sequence 3 of head 1 has no S0 member
        g["arg_ret"][1, 331], g["best_ret"][1, 331] = 5, 0.0
    elif mistake == "non_member":
        j = int(np.nonzero(ret[0, :300] == 0)[0][-1])
        g["arg_ret"][0, i] = j
    elif mistake == "value_off":
        g["best_all"][0, i] += 3e-4
    else:                                        # the reported twin's own best made too small
        j = int(g["arg_all"][0, i])
        g["best_all"][0, j] = g["best_all"][0, i] - 1e-2
    with pytest.raises(AssertionError):
        check_every_row(K, "f32", ret, cu, w, g)

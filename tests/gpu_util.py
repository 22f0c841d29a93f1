"""Helpers shared by the GPU parity tests: moving synthetic batches to the device and
comparing HIP results with the CPU oracle under the parity protocol.

Protocol (values from the method's tolerance):
  * similarity values: |gpu - oracle| <= TOL for every row that has a candidate; rows without
    a candidate must be exactly (-1, -1) on both sides;
  * best-neighbour indices: identical, except rows whose oracle runner-up margin is < TOL
    (several neighbours are equally correct there); in that exempt class the GPU's index must
    still be a valid candidate whose oracle similarity is within TOL of the best;
  * values also stay within VALUE_BOUND (1e-4), the error bound the library's header states;
  * retained sets, token by token:
      - every orphan / donor flag that differs from the oracle's belongs to a token whose
        oracle score lies within TOL of tau;
      - the GPU's S1 must equal the repair the oracle's exact scores give under the GPU's own
        classification, except tokens whose exact score lies within TOL of that repair's
        selection cut (the rank cut is a third tie source beside tau and the runner-up);
      - that repair differs from the oracle's own S1 only when a flag differs, by at most
        four tokens per differing flag (the flipped token, the token it displaces at the cut,
        and one more swap on each side when m moves by one);
    and the logic of Sec. 3.4 replayed by the oracle on the GPU's own b must give the GPU's
    S1 and stats bit for bit.
"""
from __future__ import annotations

import json
import os

import numpy as np

import oracle

TOL = 1e-3
VALUE_BOUND = 1e-4


def to_device(keys_np, dtype: str):
    import torch
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(keys_np).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(keys_np, dtype=np.float32)).cuda()


def mask_to_device(m):
    import torch
    return torch.from_numpy(np.ascontiguousarray(m, dtype=np.uint8)).cuda()


def host(t):
    return t.detach().cpu().numpy()


def check_scores(gpu: dict, orc: dict, rows: np.ndarray, keys_np, dtype: str, retained, w: int,
                 tol: float = TOL) -> dict:
    """Compare one problem's GPU rows with the oracle's; returns exemption statistics."""
    stats = {}
    Khat = None
    for kind in ("all", "ret"):
        if "best_" + kind not in orc or gpu.get("best_" + kind) is None:
            continue
        gb = np.asarray(gpu["best_" + kind], dtype=np.float64)[rows]
        ga = np.asarray(gpu["arg_" + kind])[rows]
        ob, oa, o2 = orc["best_" + kind], orc["arg_" + kind], orc["second_" + kind]
        none = oa < 0
        assert np.all(ga[none] == -1) and np.all(gb[none] == -1.0), f"{kind}: sentinel rows differ"
        assert np.all(ga[~none] >= 0), f"{kind}: GPU reports no candidate where the oracle has one"
        v = ~none
        err = np.abs(gb[v] - ob[v])
        max_err = float(err.max()) if err.size else 0.0
        assert max_err <= tol, f"{kind}: value error {max_err}"
        assert max_err <= VALUE_BOUND, f"{kind}: value error {max_err} above the stated bound"
        exempt = v & ((ob - o2) < tol)
        mismatch = v & (ga != oa)
        bad = mismatch & ~exempt
        assert not bad.any(), f"{kind}: index mismatch outside the exempt class at rows {rows[bad][:8]}"
        em = np.flatnonzero(mismatch & exempt)
        if len(em):
            if Khat is None:
                Khat = oracle.normalise(oracle.decode_keys(keys_np, dtype))
            for r in em:
                i, j = int(rows[r]), int(ga[r])
                assert abs(i - j) > w, f"{kind}: row {i} picked j={j} inside the window"
                if kind == "ret":
                    assert retained[j], f"row {i} picked evicted j={j} for the retained reduction"
                sim = float(Khat[i] @ Khat[j])
                assert sim >= ob[r] - tol, f"{kind}: row {i} picked j={j} with sim {sim} < best {ob[r]}"
        stats[kind] = {"max_err": max_err, "rows": int(v.sum()), "exempt": int(exempt.sum()),
                       "exempt_index_diff": int(len(em))}
    return stats


def _select(b_o, cls, m, descending):
    """The m most severe members of a class under exact scores (ties by position)."""
    idx = np.flatnonzero(cls)
    key = -b_o[idx] if descending else b_o[idx]
    order = idx[np.lexsort((idx, key))]
    return order[:m], order


def _cut_exempt(b_o, gpu_taken, ref_taken, ranked, m, descending, tol):
    """Members taken by one side only must sit within tol of the exact selection's cut:
    with ranked[:m] taken, a member taken by the GPU alone scores no more than tol past the
    last taken key, one taken by the reference alone no more than tol before the first
    untaken key."""
    diff = np.flatnonzero(gpu_taken != ref_taken)
    if not len(diff):
        return 0
    assert 0 < m < len(ranked), "selection differs on a side taken whole or not at all"
    last, nxt = b_o[ranked[m - 1]], b_o[ranked[m]]
    sgn = -1.0 if descending else 1.0
    for i in diff:
        if gpu_taken[i]:
            assert sgn * (b_o[i] - last) <= tol, f"token {i} taken {b_o[i]} beyond the cut {last}"
        else:
            assert sgn * (nxt - b_o[i]) <= tol, f"token {i} left {b_o[i]} before the cut {nxt}"
    return len(diff)


def tau_f32(tau: float) -> float:
    """The threshold as the library receives it (a C float): the replay of the GPU's decisions
    compares its fp32 scores with this value, so both sides decide in the kernel's precision."""
    return float(np.float32(tau))


def replay_repair(s1_gpu, stats_gpu, b_gpu, s0, tau, n_sink, n_recent):
    """Sec. 3.4 on the GPU's own b, by the oracle: S1 and (|O|, |D|, m) bit for bit."""
    t32 = tau_f32(tau)
    r = oracle.repair(np.asarray(b_gpu, dtype=np.float64), s0, t32, n_sink, n_recent)
    s1g = np.asarray(s1_gpu).astype(bool)
    if not np.array_equal(s1g, r["s1"].astype(bool)):
        d = np.flatnonzero(s1g != r["s1"].astype(bool))
        info = [(int(i), int(np.asarray(s0)[i]), float(np.asarray(b_gpu)[i])) for i in d[:8]]
        raise AssertionError(f"logic replay differs at {len(d)} tokens (pos, s0, b): {info}; "
                             f"stats gpu {list(np.asarray(stats_gpu)[:3])} replay "
                             f"{[r['n_orphan'], r['n_donor'], r['m']]}; tau32 {t32!r}")
    assert list(np.asarray(stats_gpu)[:3]) == [r["n_orphan"], r["n_donor"], r["m"]], "stats replay differs"
    return r


def check_repair(s1_gpu, stats_gpu, b_gpu, orc: dict, s0, tau: float, n_sink: int, n_recent: int,
                 tol: float = TOL) -> dict:
    """S1 of one problem against the oracle's repair on exact scores, token by token."""
    s0 = np.asarray(s0).astype(bool)
    s1g = np.asarray(s1_gpu).astype(bool)
    b_o = np.asarray(orc["best_ret"], dtype=np.float64)
    b_g = np.asarray(b_gpu, dtype=np.float64)
    n = len(s0)
    prot = oracle.protected_mask(n, n_sink, n_recent)
    assert stats_gpu[3] == 0
    replay_repair(s1g, stats_gpu, b_g, s0, tau, n_sink, n_recent)
    # GPU classification (from its own b, in the kernel's precision) against the oracle's
    t32 = tau_f32(tau)
    O_g = ~s0 & (b_g < t32)
    D_g = s0 & ~prot & (b_g >= t32)
    O_o, D_o = orc["orphan"], orc["donor"]
    near_tau = np.abs(b_o - tau) < tol
    flips = (O_g != O_o) | (D_g != D_o)
    assert not (flips & ~near_tau).any(), f"orphan/donor flags differ away from tau at {np.flatnonzero(flips & ~near_tau)[:8]}"
    # the exact-score repair under the GPU's classification
    m_g = min(int(O_g.sum()), int(D_g.sum()))
    adm_ref, O_rank = _select(b_o, O_g, m_g, descending=False)
    ev_ref, D_rank = _select(b_o, D_g, m_g, descending=True)
    ref = s0.copy()
    ref[ev_ref] = False
    ref[adm_ref] = True
    adm_g, ev_g = s1g & ~s0, s0 & ~s1g
    ref_adm, ref_ev = ref & ~s0, s0 & ~ref
    cut_o = _cut_exempt(b_o, adm_g, ref_adm, O_rank, m_g, False, tol)
    cut_d = _cut_exempt(b_o, ev_g, ref_ev, D_rank, m_g, True, tol)
    s1o = orc["s1"].astype(bool)
    shift = int((ref != s1o).sum())
    assert shift <= 4 * int(flips.sum()), f"{shift} tokens differ from the oracle's S1 with {int(flips.sum())} flags flipped"
    exact = bool(np.array_equal(s1g, s1o))
    return {"exact": exact, "near_tau": int(near_tau.sum()), "flag_diff": int(flips.sum()),
            "cut_diff": cut_o + cut_d, "shift_diff": shift, "diff": int((s1g != s1o).sum()), "m": m_g}


def check_every_row(keys_np, dtype: str, retained, cu, w: int, gpu: dict, tol: float = VALUE_BOUND) -> dict:
    """Properties of the reported best twins that hold at any size (Sec. 3.2 Eq. 1 and the
    window; Sec. 3.4 Eq. 4), checked on every row of every problem without the O(N^2 d)
    oracle: a reported position lies outside the row's window (and in S0 for b), its
    similarity (fp64, one dot product) equals the reported value within ``tol``, the sentinel
    (-1, -1) appears exactly where no position qualifies, and, since sim(i, j) = sim(j, i),
    a row reported as the best twin of another has a best value at least that large.
    gpu holds host arrays [n_heads][T]: best_all, arg_all and, when retained is given,
    best_ret, arg_ret.  Returns counts of the rows checked."""
    H = keys_np.shape[0]
    n_rows = n_none = 0
    for h in range(H):
        for s in range(len(cu) - 1):
            a, e = int(cu[s]), int(cu[s + 1])
            n = e - a
            if n == 0:
                continue
            Kh = oracle.normalise(oracle.decode_keys(keys_np[h, a:e], dtype))
            idx = np.arange(n)
            kinds = [("all", np.ones(n, bool))]
            if retained is not None:
                kinds.append(("ret", retained[h, a:e].astype(bool)))
            for kind, mem in kinds:
                arg = np.asarray(gpu["arg_" + kind][h, a:e]).astype(np.int64)
                best = np.asarray(gpu["best_" + kind][h, a:e]).astype(np.float64)
                # members j with |i - j| > w exist iff the prefix counts outside the window are > 0
                pc = np.concatenate([[0], np.cumsum(mem)])
                lo_cnt = pc[np.clip(idx - w, 0, n)]
                hi_cnt = pc[n] - pc[np.clip(idx + w + 1, 0, n)]
                exists = (lo_cnt + hi_cnt) > 0
                has = arg >= 0
                assert np.array_equal(has, exists), f"{kind}: sentinel rows differ from rows without candidates"
                assert np.all(best[~has] == -1.0), f"{kind}: sentinel value"
                i, j = idx[has], arg[has]
                assert np.all(j < n) and np.all(np.abs(i - j) > w), f"{kind}: position inside the window"
                assert np.all(mem[j]), f"{kind}: position outside the set"
                sim = np.einsum("ij,ij->i", Kh[i], Kh[j])
                err = np.abs(sim - best[has])
                assert err.size == 0 or err.max() <= tol, f"{kind}: value at the reported position off by {err.max()}"
                n_rows += int(has.sum())
                n_none += int((~has).sum())
            ba = np.asarray(gpu["best_all"][h, a:e]).astype(np.float64)
            aa = np.asarray(gpu["arg_all"][h, a:e]).astype(np.int64)
            ok = aa >= 0
            assert np.all(ba[aa[ok]] >= ba[ok] - 2 * tol), "a reported twin has a smaller best value"
    return {"rows_with_candidate": n_rows, "rows_without": n_none}


def record_exemptions(name: str, rec: dict) -> None:
    """Print one workload's exemption accounting and, when TWINKV_PARITY_RECORD names a file,
    append it there as a JSON line (the committed parity record is made from that file)."""
    line = json.dumps({"workload": name, **rec}, sort_keys=True, default=int)
    print("PARITY", line)
    path = os.environ.get("TWINKV_PARITY_RECORD")
    if path:
        os.makedirs(os.path.dirname(os.path.abspath(path)), exist_ok=True)
        with open(path, "a") as f:
            f.write(line + "\n")


def merge_scores(agg: dict, st: dict) -> dict:
    """Sum check_scores statistics over problems (maximum of the value errors)."""
    for kind, v in st.items():
        x = agg.setdefault(kind, {"max_err": 0.0, "rows": 0, "exempt": 0, "exempt_index_diff": 0})
        x["max_err"] = max(x["max_err"], v["max_err"])
        for f in ("rows", "exempt", "exempt_index_diff"):
            x[f] += v[f]
    return agg


def merge_repairs(agg: dict, rr: dict) -> dict:
    """Sum check_repair statistics over problems."""
    agg["problems"] = agg.get("problems", 0) + 1
    agg["exact"] = agg.get("exact", 0) + int(rr["exact"])
    for f in ("near_tau", "flag_diff", "cut_diff", "shift_diff", "diff"):
        agg[f] = agg.get(f, 0) + rr[f]
    return agg

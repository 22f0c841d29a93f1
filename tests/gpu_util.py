"""Helpers shared by the GPU parity tests: moving synthetic batches to the device and
comparing HIP results with the CPU oracle under the parity protocol.

Protocol (values from the method's tolerance):
  * similarity values: |gpu - oracle| <= TOL for every row that has a candidate; rows without
    a candidate must be exactly (-1, -1) on both sides;
  * best-neighbour indices: identical, except rows whose oracle runner-up margin is < TOL
    (several neighbours are equally correct there); in that exempt class the GPU's index must
    still be a valid candidate whose oracle similarity is within TOL of the best;
  * retained sets: identical, except when a token's oracle score lies within TOL of tau or of
    a selection cut-off; then the GPU's set must be a valid repair of its own classification
    (checked property by property) and every classification difference must be such a token.
"""
from __future__ import annotations

import numpy as np

import oracle

TOL = 1e-3


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
        if "best_" + kind not in orc:
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


def check_repair(s1_gpu, stats_gpu, b_gpu, orc: dict, s0, tau: float, n_sink: int, n_recent: int,
                 tol: float = TOL) -> dict:
    """S1 of one problem against the oracle's repair on exact scores."""
    s0 = np.asarray(s0).astype(bool)
    s1g = np.asarray(s1_gpu).astype(bool)
    b_o = np.asarray(orc["best_ret"], dtype=np.float64)
    b_g = np.asarray(b_gpu, dtype=np.float64)
    n = len(s0)
    idx = np.arange(n)
    prot = (idx < n_sink) | (idx >= n - n_recent)
    # GPU classification, recomputed from the GPU's own scores
    O_g = ~s0 & (b_g < tau)
    D_g = s0 & ~prot & (b_g >= tau)
    m_g = min(int(O_g.sum()), int(D_g.sum()))
    assert list(stats_gpu[:3]) == [int(O_g.sum()), int(D_g.sum()), m_g], (stats_gpu, O_g.sum(), D_g.sum())
    assert stats_gpu[3] == 0
    # the GPU set is a valid repair of that classification
    assert s1g.sum() == s0.sum(), "budget changed"
    adm, ev = s1g & ~s0, s0 & ~s1g
    assert adm.sum() == m_g and ev.sum() == m_g
    assert not (adm & ~O_g).any() and not (ev & ~D_g).any()
    diag = oracle.exemption_diagnostics(b_o, s0, tau, n_sink, n_recent)
    near_tau = diag["tau_margin"] < tol
    O_o, D_o = orc["orphan"], orc["donor"]
    assert not ((O_g != O_o) & ~near_tau).any(), "orphan sets differ away from tau"
    assert not ((D_g != D_o) & ~near_tau).any(), "donor sets differ away from tau"
    exact = bool(np.array_equal(s1g, orc["s1"].astype(bool)))
    if not exact:
        # severity order in exact scores, up to the tolerance, on the GPU's classification
        out_o, out_d = O_g & ~adm, D_g & ~ev
        if adm.any() and out_o.any():
            assert b_o[adm].max() <= b_o[out_o].min() + 2 * tol, "orphan severity violated"
        if ev.any() and out_d.any():
            assert b_o[ev].min() >= b_o[out_d].max() - 2 * tol, "donor severity violated"
        # with no tie-class token at all, the result must be identical
        cut_vals = list(diag["orphan_cut"] or ()) + list(diag["donor_cut"] or ())
        near_cut = np.zeros(n, bool)
        for c in cut_vals:
            near_cut |= np.abs(b_o - c) < tol
        assert (near_tau | near_cut).any(), "sets differ without any near-tie token"
    return {"exact": exact, "near_tau": int(near_tau.sum()), "diff": int((s1g != orc["s1"].astype(bool)).sum()),
            "m": m_g}

"""TwinKV reference oracle -- TEST INFRASTRUCTURE ONLY.

Plain, slow, fp64 CPU implementation of what the TwinKV redundancy scorer and
repair pass compute, written from the paper ("TwinKV: A Composable Repair Pass
for KV Cache Eviction via Pairwise Key Redundancy"):

  * Sec. 3.2, Eq. 1      cosine similarity of l2-normalised keys
  * Sec. 3.2, twin rule  j is a twin of i iff sim(i,j) > tau and |i-j| > w (Eq. 2 domain)
  * Sec. 3.4, Eq. 4      b_i(S0): best similarity to a retained key outside i's window,
                         -1 when no such key exists
  * Sec. 3.4             orphans / redundant donors, severity ranking, m = min(|O|,|D|),
                         the budget-preserving swap producing S1 with |S1| = |S0|
  * Sec. 3.2, Eq. 2-3    the standalone scorer: twin counts r_i, scores s_i = -r_i / n,
                         and the retained set of the highest scores with the sink and
                         recent regions at the maximum score
  * Sec. 2 (Fig. 1b)     prevalence: how many tokens have at least one twin, per threshold
  * Sec. 3.1             the compacted cache: only the keys and values at the retained
                         positions survive eviction, gathered in position order
  * Sec. 3.4             diagnostics of the repair's decisions near a boundary: distance
                         to tau, runner-up margins and the keys at each selection cut
  * Sec. 3.1 / 3.2       the retained set of a score-based policy: the K highest scores,
                         with the sink and recent regions at the maximum score

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It shares no code with the HIP library:
it never imports ``paper_2608_27128_amd`` and the library never imports it.

Readings where the paper is silent (each is exercised by a pin test):
  R1  repair uses b < tau (orphan) and b >= tau (donor) literally (Sec. 3.4); the twin
      relation of Eq. 2 uses sim > tau.
  R2  the "no surviving twin" value is -1.0 with index -1.
  R3  a zero-norm key normalises to the zero vector, so its similarity to every key is 0.
  R4  non-finite key values are an error.
  R5  argmax ties resolve to the smallest j.
  R6  severity ties resolve by ascending position (orphans: b ascending then index
      ascending; donors: b descending then index ascending).
  R11 the swap is one simultaneous pass against S0; b is not recomputed between swaps.
  R16 w >= 0, which makes the paper's extra j != i condition implied by |i-j| > w.
  R19 the scorer's budget K is given directly (the paper's ceil((1-rho) n) is the caller's);
      among equal scores the later position is retained first (recency).
  R20 the protected regions take the maximum score, so with K >= |P| they are all kept;
      with K < |P| the same order (later position first) decides among them.
  R22 a wrapped policy's retained set from its per-token scores (Sec. 3.1 selects |S| = K
      positions per head and layer; Sec. 3.2 gives the protected regions the maximum
      score): protected positions first, then higher scores; equal scores and the
      protected positions among themselves go to the lower position first; a NaN score
      ranks below every number, and -0 equals +0.
  R21 compaction writes the kept rows of each problem in ascending position order into
      `capacity` reserved rows; rows past the kept count are zero with position -1, and
      a problem that keeps more positions than it has rows is an error (status 1) whose
      rows are all zero with position -1.
Indices are 0-based positions within a sequence (the paper's 1-based positions only
enter through |i-j| and region sizes, which the shift does not change).

Parity status: every function below is pinned by tests under tests/ (closed forms,
hand-derived cases, invariants, planted-mutation checks); none is "parity unpinned".
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "decode_keys", "normalise", "similarity_rows", "window_domain", "best_twin",
    "nn_scores", "classify", "rank_severity", "repair", "repair_problem",
    "protected_mask", "twin_counts", "redundancy_scores", "evict_by_score",
    "score_evict_problem", "prevalence", "compact_problem", "compact",
    "exemption_diagnostics", "select_topk",
]

# Rows of the similarity matrix are evaluated in independent groups so that an
# (rows x n) fp64 slab stays below this many elements; each row's result does not
# depend on the grouping.
_SLAB_ELEMS = 1 << 25


# ----------------------------------------------------------------------------
# Inputs
# ----------------------------------------------------------------------------
def decode_keys(keys: np.ndarray, dtype: str) -> np.ndarray:
    """Exact fp64 values of stored keys: raw bf16 bits (uint16) or float32.  (R4: non-finite -> error)"""
    if dtype == "bf16":
        k = (np.asarray(keys, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)
    elif dtype == "f32":
        k = np.asarray(keys, dtype=np.float32)
    else:
        raise ValueError(f"unsupported key dtype {dtype!r}")
    k = k.astype(np.float64)
    if not np.all(np.isfinite(k)):
        raise ValueError("non-finite key value")
    return k


# ----------------------------------------------------------------------------
# Sec. 3.2: normalisation and Eq. 1
# ----------------------------------------------------------------------------
def normalise(K: np.ndarray) -> np.ndarray:
    """k_hat_i = k_i / ||k_i||_2 (Sec. 3.2); a zero key stays zero (reading R3)."""
    norm = np.sqrt(np.sum(K * K, axis=1))
    out = np.zeros_like(K)
    nz = norm > 0
    out[nz] = K[nz] / norm[nz, None]
    return out


def similarity_rows(Khat: np.ndarray, rows: np.ndarray) -> np.ndarray:
    """sim(i, j) = k_hat_i^T k_hat_j for the requested rows i and all j (Eq. 1)."""
    return Khat[rows] @ Khat.T


def window_domain(rows: np.ndarray, n: int, w: int, member: np.ndarray | None = None) -> np.ndarray:
    """Valid (i, j) pairs: |i - j| > w (twin rule, Sec. 3.2 / Eq. 4), optionally j in S0."""
    j = np.arange(n)
    valid = np.abs(rows[:, None] - j[None, :]) > w
    if member is not None:
        valid &= member[None, :].astype(bool)
    return valid


def best_twin(S: np.ndarray, valid: np.ndarray):
    """Row-wise max / argmax of S over valid entries, plus the runner-up value.

    Argmax ties go to the smallest j (R5).  Rows with no valid entry get (-1.0, -1)
    (R2, Eq. 4).  The runner-up is the second largest value over the valid entries
    (equal to the best when the best is attained twice); -inf when fewer than two
    entries are valid.  It is used only to report how close a row is to a tie.
    """
    n_rows, n = S.shape
    M = np.where(valid, S, -np.inf)
    any_valid = valid.any(axis=1)
    arg = np.argmax(M, axis=1)                     # first maximal index = smallest j
    best = M[np.arange(n_rows), arg]
    M[np.arange(n_rows), arg] = -np.inf            # the runner-up: best of the remaining entries
    second = M.max(axis=1) if n >= 2 else np.full(n_rows, -np.inf)
    best = np.where(any_valid, best, -1.0)
    arg = np.where(any_valid, arg, -1).astype(np.int64)
    return best, arg, second


def nn_scores(keys: np.ndarray, dtype: str, retained: np.ndarray | None, w: int,
              rows: np.ndarray | None = None) -> dict:
    """Best twin of each requested row over all keys and over the retained set.

    best_all / arg_all : max / argmax over j with |i-j| > w of sim(i, j)
                         (the twin search of Sec. 3.2 reduced to its best candidate;
                         best_all > tau iff token i has at least one twin, Eq. 2)
    best_ret / arg_ret : b_i(S0) of Eq. 4 -- the same over j in S0
    second_*           : runner-up values (diagnostic)
    """
    if w < 0:
        raise ValueError("w must be >= 0")
    K = decode_keys(keys, dtype)
    n = K.shape[0]
    Khat = normalise(K)
    rows = np.arange(n) if rows is None else np.asarray(rows, dtype=np.int64)
    out = {k: np.empty(len(rows)) for k in ("best_all", "second_all", "best_ret", "second_ret")}
    out["arg_all"] = np.empty(len(rows), dtype=np.int64)
    out["arg_ret"] = np.empty(len(rows), dtype=np.int64)
    step = max(1, _SLAB_ELEMS // max(n, 1))
    for a in range(0, len(rows), step):
        r = rows[a:a + step]
        S = similarity_rows(Khat, r)
        b, g, s2 = best_twin(S, window_domain(r, n, w))
        out["best_all"][a:a + step], out["arg_all"][a:a + step], out["second_all"][a:a + step] = b, g, s2
        if retained is not None:
            b, g, s2 = best_twin(S, window_domain(r, n, w, member=retained))
            out["best_ret"][a:a + step], out["arg_ret"][a:a + step], out["second_ret"][a:a + step] = b, g, s2
    if retained is None:
        for k in ("best_ret", "second_ret", "arg_ret"):
            del out[k]
    return out


# ----------------------------------------------------------------------------
# Sec. 3.4: composable repair
# ----------------------------------------------------------------------------
def protected_mask(n: int, n_sink: int, n_recent: int) -> np.ndarray:
    """Leading n_sink sink tokens and trailing n_recent recent tokens (Sec. 3.2 / 3.4)."""
    idx = np.arange(n)
    return (idx < n_sink) | (idx >= n - n_recent)


def classify(b: np.ndarray, s0: np.ndarray, tau: float, n_sink: int, n_recent: int):
    """Orphans: i not in S0 with b_i < tau.  Donors: j in S0, outside the protected
    regions, with b_j >= tau (Sec. 3.4, reading R1)."""
    s0 = np.asarray(s0).astype(bool)
    b = np.asarray(b, dtype=np.float64)
    prot = protected_mask(len(b), n_sink, n_recent)
    orphan = ~s0 & (b < tau)
    donor = s0 & ~prot & (b >= tau)
    return orphan, donor


def rank_severity(b: np.ndarray, orphan: np.ndarray, donor: np.ndarray):
    """Orphans by ascending b, donors by descending b (Sec. 3.4); ties by position (R6)."""
    b = np.asarray(b, dtype=np.float64)
    O = np.flatnonzero(orphan)
    D = np.flatnonzero(donor)
    O = O[np.lexsort((O, b[O]))]
    D = D[np.lexsort((D, -b[D]))]
    return O, D


def repair(b: np.ndarray, s0: np.ndarray, tau: float, n_sink: int, n_recent: int) -> dict:
    """One repair pass (Sec. 3.4): swap the m = min(|O|, |D|) most severe pairs.

    Each swap evicts a redundant donor and admits an orphan, so |S1| = |S0| (R11: one
    simultaneous pass against S0).  Returns S1 (uint8), the sets and the ranked lists.
    """
    s0 = np.asarray(s0).astype(bool)
    orphan, donor = classify(b, s0, tau, n_sink, n_recent)
    O, D = rank_severity(b, orphan, donor)
    m = min(len(O), len(D))
    s1 = s0.copy()
    s1[D[:m]] = False
    s1[O[:m]] = True
    assert s1.sum() == s0.sum()
    return {"s1": s1.astype(np.uint8), "orphan": orphan, "donor": donor,
            "n_orphan": len(O), "n_donor": len(D), "m": m,
            "orphans_ranked": O, "donors_ranked": D}


def exemption_diagnostics(b: np.ndarray, s0: np.ndarray, tau: float, n_sink: int,
                          n_recent: int, second: np.ndarray | None = None) -> dict:
    """Where the repair's discrete decisions sit close to a boundary (for accounting the
    tokens a floating-point scorer may legitimately classify or rank differently):
    |b_i - tau| (orphan / donor tests, Sec. 3.4), b_i - runner-up (the best-twin index),
    and the keys on both sides of each selection cut, b(O[m-1]) and b(O[m]) for the orphans
    and b(D[m-1]) and b(D[m]) for the donors, when that side is cut (m below its size)."""
    b = np.asarray(b, dtype=np.float64)
    r = repair(b, s0, tau, n_sink, n_recent)
    O, D, m = r["orphans_ranked"], r["donors_ranked"], r["m"]
    out = {"tau_margin": np.abs(b - tau),
           "orphan_cut": (float(b[O[m - 1]]), float(b[O[m]])) if 0 < m < len(O) else None,
           "donor_cut": (float(b[D[m - 1]]), float(b[D[m]])) if 0 < m < len(D) else None}
    if second is not None:
        out["runner_up_margin"] = b - np.asarray(second, dtype=np.float64)
    return out


def repair_problem(keys: np.ndarray, dtype: str, s0: np.ndarray, budget: int, tau: float,
                   w: int, n_sink: int, n_recent: int) -> dict:
    """Full path for one (sequence, layer, KV head) problem: Eq. 4 scores, then repair.

    The budget must equal |S0| (Sec. 3.4: the pass needs K = |S| and S0).
    """
    s0 = np.asarray(s0).astype(bool)
    if int(s0.sum()) != int(budget):
        raise ValueError(f"budget {budget} != |S0| = {int(s0.sum())}")
    sc = nn_scores(keys, dtype, s0.astype(np.uint8), w)
    out = repair(sc["best_ret"], s0, tau, n_sink, n_recent)
    out.update(sc)
    return out


# ----------------------------------------------------------------------------
# Sec. 3.2, Eq. 2-3: the standalone scorer
# ----------------------------------------------------------------------------
def twin_counts(keys: np.ndarray, dtype: str, tau: float, w: int,
                rows: np.ndarray | None = None, margin: float = 0.0) -> dict:
    """Eq. 2: r_i = #{ j : |i - j| > w, sim(i, j) > tau } for the requested rows.

    With margin > 0, also the counts at tau + margin and tau - margin: bounds on what a
    computation whose similarities are within margin of these can report.
    """
    if w < 0:
        raise ValueError("w must be >= 0")
    K = decode_keys(keys, dtype)
    n = K.shape[0]
    Khat = normalise(K)
    rows = np.arange(n) if rows is None else np.asarray(rows, dtype=np.int64)
    out = {"counts": np.zeros(len(rows), dtype=np.int64)}
    if margin > 0:
        out["counts_lo"] = np.zeros(len(rows), dtype=np.int64)
        out["counts_hi"] = np.zeros(len(rows), dtype=np.int64)
    step = max(1, _SLAB_ELEMS // max(n, 1))
    for a in range(0, len(rows), step):
        r = rows[a:a + step]
        S = similarity_rows(Khat, r)
        valid = window_domain(r, n, w)
        out["counts"][a:a + step] = np.sum(valid & (S > tau), axis=1)
        if margin > 0:
            out["counts_lo"][a:a + step] = np.sum(valid & (S > tau + margin), axis=1)
            out["counts_hi"][a:a + step] = np.sum(valid & (S > tau - margin), axis=1)
    return out


def redundancy_scores(counts: np.ndarray, n: int) -> np.ndarray:
    """Eq. 3: s_i = -r_i / n (fewer twins, higher score)."""
    return -np.asarray(counts, dtype=np.float64) / float(n)


def evict_by_score(counts: np.ndarray, budget: int, n_sink: int, n_recent: int) -> np.ndarray:
    """The retained set of Sec. 3.2: the `budget` highest scores, the sink and recent
    regions at the maximum score (R20), equal scores resolved toward the later position
    (R19).  Returns a uint8 mask."""
    counts = np.asarray(counts, dtype=np.int64)
    n = len(counts)
    if budget < 0:
        raise ValueError("budget must be >= 0")
    score = np.where(protected_mask(n, n_sink, n_recent), np.inf, redundancy_scores(counts, n))
    pos = np.arange(n)
    order = np.lexsort((-pos, -score))     # score descending, then position descending
    keep = np.zeros(n, dtype=np.uint8)
    keep[order[:min(budget, n)]] = 1
    return keep


def select_topk(scores: np.ndarray, budget: int, n_sink: int, n_recent: int) -> np.ndarray:
    """The retained set of a score-based policy (Sec. 3.1: |S| = K positions kept per head
    and layer; Sec. 3.2: the sink and recent regions take the maximum score): the `budget`
    best positions in the order of reading R22.  Returns a uint8 mask."""
    sc = np.asarray(scores, dtype=np.float64)
    n = len(sc)
    if budget < 0:
        raise ValueError("budget must be >= 0")
    prot = protected_mask(n, n_sink, n_recent)
    # the protected positions all take the maximum score (so they tie among themselves);
    # comparisons treat -0 and +0 as equal
    nan = np.isnan(sc) & ~prot
    s = np.where(prot, np.inf, np.where(nan, 0.0, sc))
    pos = np.arange(n)
    # ascending sort keys, last one primary: protected first, non-NaN before NaN,
    # higher score first, lower position first
    order = np.lexsort((pos, -s, nan, ~prot))
    keep = np.zeros(n, dtype=np.uint8)
    keep[order[:min(budget, n)]] = 1
    return keep


def score_evict_problem(keys: np.ndarray, dtype: str, budget: int, tau: float, w: int,
                        n_sink: int, n_recent: int) -> dict:
    """The scorer of Sec. 3.2 on one (sequence, layer, KV head) problem: Eq. 2 counts,
    Eq. 3 scores and the retained set."""
    c = twin_counts(keys, dtype, tau, w)["counts"]
    n = len(c)
    return {"counts": c, "scores": redundancy_scores(c, n),
            "retained": evict_by_score(c, budget, n_sink, n_recent)}


# ----------------------------------------------------------------------------
# Sec. 2, Fig. 1b: prevalence of twins
# ----------------------------------------------------------------------------
def prevalence(best_all: np.ndarray, taus) -> np.ndarray:
    """Number of tokens with at least one twin for each threshold: a token has a twin at
    tau exactly when its best similarity outside the window exceeds tau (Eq. 2), and a
    token without any candidate (best = -1, reading R2) has none for tau >= -1."""
    b = np.asarray(best_all, dtype=np.float64)
    return np.array([int(np.sum(b > float(t))) for t in taus], dtype=np.int64)


# ----------------------------------------------------------------------------
# Sec. 3.1: the compacted cache
# ----------------------------------------------------------------------------
def compact_problem(keys: np.ndarray, values: np.ndarray | None, retained: np.ndarray,
                    capacity: int) -> dict:
    """One (sequence, layer, KV head) problem: eviction keeps only the keys and values at the
    retained positions (Sec. 3.1).  Rows are copied bit for bit (any element dtype), in
    ascending position order, into `capacity` rows (reading R21)."""
    keys = np.asarray(keys)
    keep = np.flatnonzero(np.asarray(retained) != 0)
    n_keep = len(keep)
    if capacity < 0:
        raise ValueError("capacity must be >= 0")
    ok = n_keep <= capacity
    k_out = np.zeros((capacity,) + keys.shape[1:], dtype=keys.dtype)
    v_out = None if values is None else np.zeros((capacity,) + np.asarray(values).shape[1:],
                                                 dtype=np.asarray(values).dtype)
    pos = np.full(capacity, -1, dtype=np.int64)
    if ok:
        k_out[:n_keep] = keys[keep]
        if values is not None:
            v_out[:n_keep] = np.asarray(values)[keep]
        pos[:n_keep] = keep
    return {"keys": k_out, "values": v_out, "pos": pos,
            "stats": np.array([n_keep, capacity, 0 if ok else 1, 0], dtype=np.int64)}


def compact(keys: np.ndarray, values: np.ndarray | None, retained: np.ndarray,
            cu_seqlens, capacity) -> dict:
    """A batch [n_heads][T][...] of ragged sequences: problem (h, s) goes to rows
    [c_s, c_s + capacity[s]) of head h's block of sum(capacity) rows, c_s = sum of the
    capacities before s."""
    keys = np.asarray(keys)
    H = keys.shape[0]
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    cap = np.asarray(capacity, dtype=np.int64)
    n_seqs = len(cu) - 1
    c0 = np.concatenate([[0], np.cumsum(cap)])
    C = int(c0[-1])
    k_out = np.zeros((H, C) + keys.shape[2:], dtype=keys.dtype)
    v_out = None if values is None else np.zeros((H, C) + np.asarray(values).shape[2:],
                                                 dtype=np.asarray(values).dtype)
    pos = np.full((H, C), -1, dtype=np.int64)
    stats = np.zeros((H * n_seqs, 4), dtype=np.int64)
    for h in range(H):
        for s in range(n_seqs):
            a, e = int(cu[s]), int(cu[s + 1])
            r = compact_problem(keys[h, a:e], None if values is None else np.asarray(values)[h, a:e],
                                np.asarray(retained)[h, a:e], int(cap[s]))
            k_out[h, c0[s]:c0[s + 1]] = r["keys"]
            if values is not None:
                v_out[h, c0[s]:c0[s + 1]] = r["values"]
            pos[h, c0[s]:c0[s + 1]] = r["pos"]
            stats[h * n_seqs + s] = r["stats"]
    return {"keys": k_out, "values": v_out, "pos": pos, "stats": stats}

"""Edge cases of the repair pass's selection (Sec. 3.4: the m most severe orphans and donors):
cut-side scores that are all equal, that differ only in their last bits, that take two values
with m falling exactly at the end of the first, that form two clusters with m falling exactly
at the end of the first (whose scores differ in their low 12 bits, so the bucket of the m-th
key holds many distinct keys when the selection stops early), and that span both signs.  The
selection skips the leading bits the cut side's keys share and stops once the m-th key's
bucket is taken whole; every case must still give the oracle's S1 and counts bit for bit, for
each kernel (up to 4096 tokens, up to 16384, up to 32768, longer).  The degenerate cases, where
m = 0 and nothing may move, are covered on every kernel too."""
import numpy as np
import pytest

import oracle
from gpu_util import host, mask_to_device
from paper_2608_27128_amd import binding

pytestmark = pytest.mark.gpu

TAU = 0.5
N_SINK, N_RECENT = 4, 16
KINDS = ("equal", "lowbits", "two", "cluster", "spread")


def cut_values(kind, side, k, g):
    """k scores for the cut side (orphans: below TAU; donors: at or above it)."""
    base = np.float32(0.25 if side == "o" else 0.75)
    if kind == "equal":
        return np.full(k, base, np.float32)
    if kind == "lowbits":
        return (base.view(np.int32) + g.integers(0, 8, k).astype(np.int32)).view(np.float32)
    if kind == "two":
        hi = np.float32(0.375 if side == "o" else 0.875)
        v = np.full(k, hi, np.float32)
        v[: k // 2] = base
        return v
    if side == "o":  # spread: both signs below TAU
        return g.uniform(-1.0, TAU, k).astype(np.float32)
    return g.uniform(TAU, 1.0, k).astype(np.float32)


def make_problem(n, kind, side, g):
    """Scores b and retained set S0 of one problem whose cut side is `side` (o: orphans are
    cut, so there are fewer donors; d: the reverse)."""
    B = (4 * n) // 10
    perm = g.permutation(n)
    s0 = np.zeros(n, np.uint8)
    s0[perm[:B]] = 1
    ret = np.flatnonzero(s0)
    out = np.flatnonzero(s0 == 0)
    b = np.empty(n, np.float32)
    # defaults: retained tokens below TAU (kept, not donors), evicted ones at or above (not
    # orphans)
    b[ret] = g.uniform(0.0, TAU - 0.01, ret.size).astype(np.float32)
    b[out] = g.uniform(TAU + 0.01, 1.0, out.size).astype(np.float32)
    orph = g.permutation(out)
    # donors only outside the protected sink and recent regions, so that m is what is set here
    don = g.permutation(ret[(ret >= N_SINK) & (ret < n - N_RECENT)])
    if side == "o":
        orph = orph[: (6 * out.size) // 10]
        n_don = max(1, orph.size // 2 if kind in ("two", "cluster") else orph.size // 7)
        don = don[:n_don]
        b[orph] = g.permutation(cut_values(kind, "o", orph.size, g))
        b[don] = g.uniform(TAU, 1.0, don.size).astype(np.float32)
        if kind in ("two", "cluster"):  # m equal to the count of the lower group
            low = np.full(orph.size, np.float32(0.25))
            if kind == "cluster":  # the lower group differs in its low 12 bits
                low = (low.view(np.int32) + g.integers(0, 4096, orph.size).astype(np.int32)
                       ).view(np.float32)
            b[orph] = np.where(np.arange(orph.size) < don.size, low, np.float32(0.375))
    else:
        don = don[: (6 * ret.size) // 10]
        n_orph = max(1, don.size // 2 if kind in ("two", "cluster") else don.size // 7)
        orph = orph[:n_orph]
        b[don] = g.permutation(cut_values(kind, "d", don.size, g))
        b[orph] = g.uniform(-1.0, TAU - 0.01, orph.size).astype(np.float32)
        if kind in ("two", "cluster"):  # donors go in descending order: the higher group
            high = np.full(don.size, np.float32(0.875))
            if kind == "cluster":
                high = (high.view(np.int32) + g.integers(0, 4096, don.size).astype(np.int32)
                        ).view(np.float32)
            b[don] = np.where(np.arange(don.size) < orph.size, high, np.float32(0.75))
    return b, s0, B


@pytest.mark.parametrize("n", [3000, 9000, 30000, 40000],
                         ids=["short", "reg16", "reg32", "streaming"])
def test_selection_edges_vs_oracle(n):
    import torch
    g = np.random.default_rng(n)
    cases = [(kind, side) for kind in KINDS for side in ("o", "d")]
    H = len(cases)
    cu = np.array([0, n], np.int64)
    b = np.zeros((H, n), np.float32)
    s0 = np.zeros((H, n), np.uint8)
    budget = None
    for h, (kind, side) in enumerate(cases):
        b[h], s0[h], budget = make_problem(n, kind, side, g)
    out = binding.repair_from_scores(torch.from_numpy(b).cuda(), mask_to_device(s0), [budget],
                                     TAU, N_SINK, N_RECENT, cu)
    s1 = host(out["s1"])
    st = host(out["stats"]).reshape(H, 4)
    for h, (kind, side) in enumerate(cases):
        r = oracle.repair(b[h].astype(np.float64), s0[h], TAU, N_SINK, N_RECENT)
        assert r["m"] > 0, (kind, side)
        assert (r["n_orphan"] > r["m"]) == (side == "o"), (kind, side)
        assert np.array_equal(s1[h], r["s1"]), (kind, side)
        assert st[h].tolist() == [r["n_orphan"], r["n_donor"], r["m"], 0], (kind, side)


def run_vs_oracle(b, s0, budget, tau, n_sink, n_recent):
    import torch
    H, n = b.shape
    out = binding.repair_from_scores(torch.from_numpy(b).cuda(), mask_to_device(s0), [budget],
                                     tau, n_sink, n_recent, np.array([0, n], np.int64))
    s1, st = host(out["s1"]), host(out["stats"]).reshape(H, 4)
    for h in range(H):
        r = oracle.repair(b[h].astype(np.float64), s0[h], tau, n_sink, n_recent)
        assert np.array_equal(s1[h], r["s1"]), h
        assert st[h].tolist() == [r["n_orphan"], r["n_donor"], r["m"], 0], h
    return s1, st


@pytest.mark.parametrize("n", [3000, 9000, 30000, 40000],
                         ids=["short", "reg16", "reg32", "streaming"])
def test_degenerate_sets_vs_oracle(n):
    """Cases where nothing may move (Sec. 3.4: m = min(|O|, |D|) = 0): S0 empty (budget 0, no
    donors), S0 holding every position (no orphans), every position protected (no donors),
    and tau above or below every score; on each K3 kernel S1 must equal S0 and the counts
    the oracle's."""
    g = np.random.default_rng(n + 1)
    H = 3
    b = g.uniform(-1.0, 1.0, (H, n)).astype(np.float32)
    half = np.zeros((H, n), np.uint8)
    for h in range(H):
        half[h, g.permutation(n)[: n // 2]] = 1
    s0_none = np.zeros((H, n), np.uint8)
    s0_all = np.ones((H, n), np.uint8)
    cases = [(s0_none, 0, 0.5, N_SINK, N_RECENT), (s0_all, n, 0.5, N_SINK, N_RECENT),
             (half, n // 2, 0.5, n // 2, n - n // 2), (half, n // 2, 1.5, N_SINK, N_RECENT),
             (half, n // 2, -1.5, N_SINK, N_RECENT)]
    for s0, budget, tau, ns, nr in cases:
        s1, st = run_vs_oracle(b, s0, budget, tau, ns, nr)
        assert np.array_equal(s1, s0), (budget, tau, ns, nr)
        assert np.all(st[:, 2] == 0), (budget, tau, ns, nr)

"""The standalone scorer (Sec. 3.2, Eq. 2-3) and the prevalence statistic (Sec. 2, Fig. 1b):
HIP path vs the CPU oracle through the C ABI.

Protocol.  Twin counts are integers decided by sim > tau on fp32 similarities whose error is
below COUNT_MARGIN (fp32 accumulation of exact bf16 products; the row pre-scaling is exact).
So the GPU count of every row must lie between the oracle's counts at tau + COUNT_MARGIN and
at tau - COUNT_MARGIN, and must equal the oracle's count for every row without a pair that
close to tau.  The eviction and the prevalence take integer / threshold decisions on the GPU's
own counts and scores: replaying the oracle's logic on those must reproduce the GPU's result
bit for bit; end to end the sets must agree whenever no count was ambiguous."""
import numpy as np
import pytest

import oracle
from gpu_util import host, to_device
from paper_2608_27128_amd import binding, synth

pytestmark = pytest.mark.gpu

COUNT_MARGIN = 2e-5


def small_spec(H, lens, d, dtype, w, seed, dup_frac=0.25, sigma=0.02, recipe="offset"):
    return synth.Spec(name="scorer", config_id=80 + seed, n_heads=H, lens=tuple(lens), d=d,
                      dtype=dtype, key_recipe=recipe, dup_recipe="uniform", dup_frac=dup_frac,
                      dup_sigma=sigma, budget_frac=0.5, policy_sinks=4, policy_recent=8,
                      tau=0.9, w=w, n_sink=4, n_recent=8, seed=seed)


def check_counts(batch, gpu_counts, tau, w, rows_of=None):
    """Interval check of every (sampled) row; returns (rows, ambiguous rows, exact rows)."""
    n_rows = n_amb = n_exact = 0
    for h in range(batch.n_heads):
        for s in range(batch.n_seqs):
            a, e = int(batch.cu_seqlens[s]), int(batch.cu_seqlens[s + 1])
            if e == a:
                continue
            rows = np.arange(e - a) if rows_of is None else rows_of(h, s, e - a)
            o = oracle.twin_counts(batch.keys[h, a:e], batch.dtype, tau, w, rows=rows,
                                   margin=COUNT_MARGIN)
            g = gpu_counts[h, a:e][rows]
            assert np.all(g >= o["counts_lo"]) and np.all(g <= o["counts_hi"]), (h, s)
            amb = o["counts_lo"] != o["counts_hi"]
            assert np.array_equal(g[~amb], o["counts"][~amb]), (h, s)
            n_rows += len(rows)
            n_amb += int(amb.sum())
            n_exact += int((g == o["counts"]).sum())
    return n_rows, n_amb, n_exact


CASES = [
    # (heads, lens, d, dtype, w, tau)
    (1, [700], 64, "bf16", 32, 0.9),
    (3, [1100], 128, "bf16", 32, 0.85),
    (9, [600], 128, "bf16", 0, 0.95),           # 9 heads: the XCD-affine schedule
    (2, [1500], 64, "bf16", 128, 0.8),
    (1, [512], 64, "f32", 32, 0.9),
    (2, [333], 128, "f32", 5, 0.5),
    (3, [1, 2, 33, 34, 0, 513, 1030], 128, "bf16", 32, 0.9),   # ragged, incl. empty
    (8, [65, 700, 31], 64, "bf16", 16, 0.9),
    (1, [40], 128, "bf16", 39, 0.9),             # N <= w + 1: no candidate, every count 0
    (2, [400], 64, "bf16", 4, -0.2),             # negative tau: most pairs count
]


@pytest.mark.parametrize("H,lens,d,dtype,w,tau", CASES)
def test_twin_counts_vs_oracle(H, lens, d, dtype, w, tau):
    seed = (H * 131 + sum(lens) * 7 + d + w) % 997
    batch = synth.make_batch(small_spec(H, lens, d, dtype, w, seed))
    out = binding.twin_counts(to_device(batch.keys, dtype), tau, w, batch.cu_seqlens)
    assert np.all(host(out["status"]) == 0)
    counts = host(out["counts"])
    n, amb, exact = check_counts(batch, counts, tau, w)
    print("twin counts", H, lens, d, dtype, w, tau, "rows", n, "ambiguous", amb, "exact", exact)
    if lens == [40] and w == 39:
        assert np.all(counts == 0)


def test_counts_agree_with_best_twin():
    """r_i >= 1 exactly when best_all_i > tau (two independent GPU paths), away from tau."""
    batch = synth.make_batch(small_spec(4, [1200, 800], 128, "bf16", 32, 21))
    kt = to_device(batch.keys, "bf16")
    tau = 0.9
    c = host(binding.twin_counts(kt, tau, 32, batch.cu_seqlens)["counts"])
    b = host(binding.nn_scores(kt, None, 32, batch.cu_seqlens)["best_all"])
    far = np.abs(b - tau) > 1e-4
    assert np.array_equal((c >= 1)[far], (b > tau)[far])


def replay_evict(batch, gpu, budget, n_sink, n_recent):
    """Bit-exact logic replay of the eviction (and of Eq. 3) on the GPU's own counts."""
    kept, cnt, sc = host(gpu["retained"]), host(gpu["counts"]), host(gpu["scores"])
    st = host(gpu["stats"]).reshape(batch.n_heads, batch.n_seqs, 4)
    for h in range(batch.n_heads):
        for s in range(batch.n_seqs):
            a, e = int(batch.cu_seqlens[s]), int(batch.cu_seqlens[s + 1])
            n = e - a
            b = int(np.broadcast_to(budget, (batch.n_seqs,))[s])
            want = oracle.evict_by_score(cnt[h, a:e], b, n_sink, n_recent)
            assert np.array_equal(kept[h, a:e], want), (h, s)
            assert st[h, s, 0] == min(b, n) and st[h, s, 2] == 0
            if n:
                np.testing.assert_allclose(sc[h, a:e], oracle.redundancy_scores(cnt[h, a:e], n),
                                           rtol=1e-6, atol=0)


@pytest.mark.parametrize("H,lens,d,dtype,w,tau,budget_frac,n_sink,n_recent", [
    (3, [1100], 128, "bf16", 32, 0.85, 0.5, 4, 64),
    (2, [900, 350], 64, "bf16", 32, 0.9, 0.3, 4, 0),
    (9, [700], 128, "bf16", 16, 0.9, 0.7, 4, 16),
    (2, [300], 64, "f32", 8, 0.8, 0.5, 2, 3),
    (3, [1, 2, 33, 0, 513], 128, "bf16", 32, 0.9, 0.5, 4, 8),
])
def test_score_evict_vs_oracle(H, lens, d, dtype, w, tau, budget_frac, n_sink, n_recent):
    seed = (H * 17 + sum(lens) + w) % 991
    batch = synth.make_batch(small_spec(H, lens, d, dtype, w, seed))
    budget = np.array([int(np.floor(budget_frac * L)) for L in lens], dtype=np.int64)
    gpu = binding.score_evict(to_device(batch.keys, dtype), budget, tau, w, n_sink, n_recent,
                              batch.cu_seqlens)
    replay_evict(batch, gpu, budget, n_sink, n_recent)
    check_counts(batch, host(gpu["counts"]), tau, w)
    # end to end: problems whose oracle counts equal the GPU's give the same kept set
    kept, cnt = host(gpu["retained"]), host(gpu["counts"])
    same = 0
    for h in range(H):
        for s in range(len(lens)):
            a, e = int(batch.cu_seqlens[s]), int(batch.cu_seqlens[s + 1])
            o = oracle.score_evict_problem(batch.keys[h, a:e], dtype, int(budget[s]), tau, w,
                                           n_sink, n_recent)
            if np.array_equal(o["counts"], cnt[h, a:e]):
                assert np.array_equal(o["retained"], kept[h, a:e]), (h, s)
                same += 1
    print("score_evict problems with identical counts:", same, "of", H * len(lens))
    assert same >= (H * len(lens)) // 2


@pytest.mark.parametrize("n", [4096, 4097, 9000, 16384, 16385, 20000, 32768, 32769, 40000])
def test_score_evict_every_cache_size(n):
    """The eviction kernel keeps an LDS copy of the counts for sequences of up to 4096, 16384
    and 32768 tokens and reads global memory beyond that; the logic replay on the GPU's own
    counts must hold bit for bit in every variant, at each limit and one token past it."""
    batch = synth.make_batch(small_spec(1, [n], 64, "bf16", 32, 7 + n % 97, dup_frac=0.3))
    budget = np.array([(3 * n) // 10], dtype=np.int64)
    gpu = binding.score_evict(to_device(batch.keys, "bf16"), budget, 0.8, 32, 4, 64,
                              batch.cu_seqlens)
    replay_evict(batch, gpu, budget, 4, 64)


def test_score_evict_budget_edges():
    """Budget 0, below the protected regions, at and above the length."""
    batch = synth.make_batch(small_spec(2, [100, 120, 90, 60], 64, "bf16", 8, 31))
    kt = to_device(batch.keys, "bf16")
    budget = np.array([0, 5, 90, 200], dtype=np.int64)      # 5 < |P| = 4 + 8
    gpu = binding.score_evict(kt, budget, 0.9, 8, 4, 8, batch.cu_seqlens)
    replay_evict(batch, gpu, budget, 4, 8)
    kept = host(gpu["retained"])
    cu = batch.cu_seqlens
    assert kept[:, cu[0]:cu[1]].sum() == 0
    assert np.all(kept[:, cu[1]:cu[2]].sum(1) == 5)
    assert np.all(kept[:, cu[1] + 115:cu[2]] == 1)          # the 5 latest recent positions
    assert np.all(kept[:, cu[2]:cu[3]] == 1) and np.all(kept[:, cu[3]:cu[4]] == 1)


def test_prevalence_vs_oracle():
    batch = synth.make_batch(small_spec(5, [1000, 300, 0, 77], 128, "bf16", 32, 41))
    kt = to_device(batch.keys, "bf16")
    out = binding.nn_scores(kt, None, 32, batch.cu_seqlens)
    taus = [0.5, 0.8, 0.85, 0.9, 0.95, 0.99, -1.0, -2.0, 1.0]
    prev = host(binding.prevalence(out["best_all"], taus, batch.cu_seqlens)).reshape(5, 4, len(taus))
    b = host(out["best_all"])
    for h in range(5):
        for s in range(4):
            a, e = int(batch.cu_seqlens[s]), int(batch.cu_seqlens[s + 1])
            # replay on the GPU's own best_all: exact
            np.testing.assert_array_equal(prev[h, s], oracle.prevalence(b[h, a:e], taus))
            if e > a:
                ob = oracle.nn_scores(batch.keys[h, a:e], "bf16", None, 32)["best_all"]
                lo = oracle.prevalence(ob, [t + 1e-4 for t in taus])
                hi = oracle.prevalence(ob, [t - 1e-4 for t in taus])
                assert np.all(prev[h, s] >= lo) and np.all(prev[h, s] <= hi)


def test_twin_counts_full_llama1b_8k():
    """The 16 x 8 x 8192 d=64 cache: sampled rows of three problems against the oracle, and the
    count / best-twin equivalence on every row of every problem."""
    batch = synth.make_batch(synth.spec("llama1b_8k"))
    sp = batch.spec
    kt = to_device(batch.keys, batch.dtype)
    counts = host(binding.twin_counts(kt, sp.tau, sp.w, batch.cu_seqlens)["counts"])
    best = host(binding.nn_scores(kt, None, sp.w, batch.cu_seqlens)["best_all"])
    far = np.abs(best - sp.tau) > 1e-4
    assert np.array_equal((counts >= 1)[far], (best > sp.tau)[far])
    rng = np.random.default_rng(5)
    picks = {(0, 0), (64, 0), (127, 0)}

    def rows_of(h, s, n):
        return np.sort(rng.choice(n, 96, replace=False))
    n, exact = 0, 0
    for (h, s) in picks:
        a, e = int(batch.cu_seqlens[s]), int(batch.cu_seqlens[s + 1])
        rows = rows_of(h, s, e - a)
        o = oracle.twin_counts(batch.keys[h, a:e], batch.dtype, sp.tau, sp.w, rows=rows,
                               margin=COUNT_MARGIN)
        g = counts[h, a:e][rows]
        assert np.all(g >= o["counts_lo"]) and np.all(g <= o["counts_hi"])
        n += len(rows)
        exact += int((g == o["counts"]).sum())
    print("llama1b_8k twin counts: sampled rows", n, "exact", exact)


def test_nonfinite_key_in_counts_and_eviction():
    """A NaN key: its problem is flagged (twin counts and the scorer), the scorer still keeps
    exactly its budget there with the protected regions first, and every other problem's
    counts and kept set equal those of the same batch without the NaN, bit for bit."""
    batch = synth.make_batch(small_spec(3, [400, 300], 128, "bf16", 16, 43))
    clean = to_device(batch.keys, "bf16")
    keys = batch.keys.copy()
    keys[2, 500, 9] = 0x7FC0                   # NaN in head 2, sequence 1
    dirty = to_device(keys, "bf16")
    cu = batch.cu_seqlens
    good = np.ones(keys.shape[:2], bool)
    good[2, cu[1]:cu[2]] = False
    c0 = binding.twin_counts(clean, 0.9, 16, cu)
    c1 = binding.twin_counts(dirty, 0.9, 16, cu)
    assert host(c1["status"]).reshape(3, 2).tolist() == [[0, 0], [0, 0], [0, 2]]
    assert np.array_equal(host(c0["counts"])[good], host(c1["counts"])[good])
    budget = np.array([150, 120], np.int64)
    e0 = binding.score_evict(clean, budget, 0.9, 16, 4, 8, cu)
    e1 = binding.score_evict(dirty, budget, 0.9, 16, 4, 8, cu)
    st = host(e1["stats"]).reshape(3, 2, 4)
    assert st[2, 1, 2] == 2 and st[:, :, 2].sum() == 2
    k0, k1 = host(e0["retained"]), host(e1["retained"])
    assert np.array_equal(k0[good], k1[good])
    bad = k1[2, cu[1]:cu[2]]
    assert bad.sum() == 120 and bad[:4].all() and bad[-8:].all()

"""A score-based policy's retained set on the GPU (Sec. 3.1: K positions per head and layer;
Sec. 3.2: the protected regions at the maximum score; reading R22 for ties, NaN and signed
zeros) against the oracle, bit for bit, and the whole pipeline scores -> S0 -> repair -> S1
-> compacted cache on the GPU against the oracle."""
import numpy as np
import pytest

import oracle
from gpu_util import check_repair, check_scores, host, mask_to_device, to_device
from paper_2608_27128_amd import binding, synth

pytestmark = pytest.mark.gpu


def draw_scores(rng, H, T, kind):
    if kind == "normal":
        return rng.standard_normal((H, T)).astype(np.float32)
    if kind == "ties":                       # a handful of values: long runs of exact ties
        return rng.integers(-3, 4, (H, T)).astype(np.float32) * 0.25
    if kind == "special":                    # signed zeros, infinities and NaN among ties
        pool = np.array([0.0, -0.0, 0.5, -0.5, np.inf, -np.inf, np.nan, 1.0], dtype=np.float32)
        return pool[rng.integers(0, len(pool), (H, T))]
    if kind == "equal":
        return np.full((H, T), 0.125, np.float32)
    raise ValueError(kind)


def run_select(scores, lens, budgets, n_sink, n_recent):
    import torch
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    out = binding.select_topk(torch.from_numpy(scores).cuda(), budgets, n_sink, n_recent, cu)
    keep, st = host(out["retained"]), host(out["stats"]).reshape(scores.shape[0], len(lens), 4)
    for h in range(scores.shape[0]):
        for s in range(len(lens)):
            a, e = int(cu[s]), int(cu[s + 1])
            want = oracle.select_topk(scores[h, a:e], int(budgets[s]), n_sink, n_recent)
            np.testing.assert_array_equal(keep[h, a:e], want, err_msg=f"head {h} seq {s}")
            nan = int(np.isnan(scores[h, a:e]).sum())
            assert st[h, s].tolist() == [min(int(budgets[s]), e - a), nan, 0, 0], (h, s)
    return keep


@pytest.mark.parametrize("kind", ["normal", "ties", "special", "equal"])
@pytest.mark.parametrize("lens", [[700], [1, 0, 33, 257, 1030], [5000], [20000], [40000]])
def test_select_topk_vs_oracle(kind, lens):
    """Every workgroup size (256 threads up to 4096 tokens, 1024 up to 16384 and 32768 with
    the LDS copy, and the uncached path beyond) and ragged batches with empty sequences."""
    rng = np.random.default_rng(len(lens) * 7 + sum(lens) + len(kind))
    H = 3
    T = int(sum(lens))
    scores = draw_scores(rng, H, T, kind)
    budgets = [int(rng.integers(0, n + 1)) if n else 0 for n in lens]
    run_select(scores, lens, budgets, 4, 64)


@pytest.mark.parametrize("n", [4096, 4097, 16384, 16385, 32768, 32769])
@pytest.mark.parametrize("kind", ["ties", "special"])
def test_select_topk_size_boundaries(n, kind):
    """The longest sequence of a batch picks the selection's workgroup size and whether the
    keys are copied to LDS (4096, 16384 and 32768 tokens): a sequence at each limit and one
    past it, with a short sequence beside it in the same batch, bit for bit."""
    rng = np.random.default_rng(n + len(kind))
    lens = [n, 37]
    scores = draw_scores(rng, 2, sum(lens), kind)
    run_select(scores, lens, [int(rng.integers(0, n + 1)), 20], 4, 64)


def test_select_topk_budget_edges():
    """Budget 0, below the protected count (the lowest protected positions), exactly the
    protected count, the length and beyond; protected regions covering everything."""
    rng = np.random.default_rng(3)
    lens = [300] * 7
    scores = draw_scores(rng, 2, sum(lens), "ties")
    run_select(scores, lens, [0, 3, 68, 150, 300, 301, 10 ** 6], 4, 64)
    run_select(scores, lens, [0, 1, 50, 299, 300, 500, 7], 200, 200)


def test_pipeline_scores_to_compacted_cache():
    """Policy scores -> S0 (select_topk) -> repair -> S1 -> compaction, all on the GPU, against
    the oracle at every step (S0 and the compacted cache exactly, the repair under the
    parity protocol)."""
    import torch
    sp = synth.Spec(name="pipeline", config_id=98, n_heads=3, lens=(900, 0, 333, 1500), d=128,
                    dtype="bf16", key_recipe="offset", dup_recipe="uniform", dup_frac=0.2,
                    dup_sigma=0.02, budget_frac=0.4, policy_sinks=4, policy_recent=32, tau=0.9,
                    w=32, n_sink=4, n_recent=32, seed=5)
    batch = synth.make_batch(sp)
    cu = batch.cu_seqlens
    H, T = batch.retained.shape
    rng = np.random.default_rng(8)
    scores = draw_scores(rng, H, T, "ties")
    sel = binding.select_topk(torch.from_numpy(scores).cuda(), batch.budget, sp.n_sink,
                              sp.n_recent, cu)
    s0 = host(sel["retained"])
    kt = to_device(batch.keys, "bf16")
    out = binding.repair(kt, sel["retained"], batch.budget, sp.tau, sp.w, sp.n_sink, sp.n_recent,
                         cu)
    s1, b = host(out["s1"]), host(out["best_ret"])
    st = host(out["stats"]).reshape(H, len(sp.lens), 4)
    gpu_all = {k: host(out[k]) for k in ("best_all", "arg_all", "best_ret", "arg_ret")}
    for h in range(H):
        for s in range(len(sp.lens)):
            a, e = int(cu[s]), int(cu[s + 1])
            if e == a:
                continue
            r = oracle.select_topk(scores[h, a:e], int(batch.budget[s]), sp.n_sink, sp.n_recent)
            np.testing.assert_array_equal(s0[h, a:e], r)
            k = batch.keys[h, a:e]
            orc = oracle.repair_problem(k, "bf16", r, batch.budget[s], sp.tau, sp.w, sp.n_sink,
                                        sp.n_recent)
            check_repair(s1[h, a:e], st[h, s], b[h, a:e], orc, r, sp.tau, sp.n_sink, sp.n_recent)
            check_scores({kk: v[h, a:e] for kk, v in gpu_all.items()}, orc, np.arange(e - a), k,
                         "bf16", r, sp.w)
    comp = binding.compact(kt, out["s1"], batch.budget, cu_seqlens=cu)
    o = oracle.compact(batch.keys, None, s1, cu, batch.budget)
    np.testing.assert_array_equal(host(comp["pos"]), o["pos"])
    np.testing.assert_array_equal(host(comp["stats"]), o["stats"])
    assert np.array_equal(host(comp["keys"].view(torch.int16)).view(np.uint16), o["keys"])

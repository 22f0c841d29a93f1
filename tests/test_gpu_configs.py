"""The five workloads at their full sizes, in the launch configuration bench.py times.

The GPU processes every problem of each workload in one call.  The oracle checks sampled
rows of sampled problems (each row costs O(N d)), complete problems where a full O(N^2 d)
oracle pass is affordable, and properties that must hold for every problem at any size."""
import numpy as np
import pytest

import oracle
from gpu_util import check_repair, check_scores, host, mask_to_device, to_device
from paper_2608_27128_amd import binding, synth

pytestmark = pytest.mark.gpu


def sample_rows(n, rng, k=192, rb=512):
    edges = [r for b in range(rb, n, rb) for r in (b - 1, b)]
    rows = set(range(min(n, 16))) | set(range(max(0, n - 16), n)) | set(edges[:32])
    rows |= set(rng.choice(n, size=min(n, k), replace=False).tolist())
    return np.array(sorted(rows), dtype=np.int64)


def check_all_problems(batch, out, tau, n_sink, n_recent):
    """Properties of every problem's result (budget, swap count, membership, protection)."""
    s1 = host(out["s1"])
    b = host(out["best_ret"])
    st = host(out["stats"]).reshape(batch.n_heads, batch.n_seqs, 4)
    assert np.all(st[..., 3] == 0)
    swapped = 0
    for s in range(batch.n_seqs):
        a, e = int(batch.cu_seqlens[s]), int(batch.cu_seqlens[s + 1])
        n = e - a
        s0 = batch.retained[:, a:e].astype(bool)
        s1s = s1[:, a:e].astype(bool)
        bb = b[:, a:e]
        idx = np.arange(n)
        prot = (idx < n_sink) | (idx >= n - n_recent)
        O = ~s0 & (bb < tau)
        D = s0 & ~prot[None, :] & (bb >= tau)
        m = np.minimum(O.sum(1), D.sum(1))
        assert np.all(s1s.sum(1) == batch.budget[s])
        assert np.all(st[:, s, 0] == O.sum(1)) and np.all(st[:, s, 1] == D.sum(1))
        assert np.all(st[:, s, 2] == m)
        adm, ev = s1s & ~s0, s0 & ~s1s
        assert np.all(adm.sum(1) == m) and np.all(ev.sum(1) == m)
        assert not (adm & ~O).any() and not (ev & ~D).any()
        assert not (s0 & prot[None, :] & ~s1s).any()
        swapped += int(m.sum())
    return swapped


def check_sampled_rows(batch, out, problems, rng, w):
    agg = {}
    for (h, s) in problems:
        a, e = int(batch.cu_seqlens[s]), int(batch.cu_seqlens[s + 1])
        k, r = batch.keys[h, a:e], batch.retained[h, a:e]
        rows = sample_rows(e - a, rng)
        orc = oracle.nn_scores(k, batch.dtype, r, w, rows=rows)
        g = {key: host(out[key][h, a:e]) for key in ("best_all", "arg_all", "best_ret", "arg_ret")}
        st = check_scores(g, orc, rows, k, batch.dtype, r, w)
        for kind, v in st.items():
            x = agg.setdefault(kind, {"max_err": 0.0, "rows": 0, "exempt": 0, "exempt_index_diff": 0})
            x["max_err"] = max(x["max_err"], v["max_err"])
            for f in ("rows", "exempt", "exempt_index_diff"):
                x[f] += v[f]
    return agg


def check_full_problems(batch, out, problems, tau, w, n_sink, n_recent):
    res = []
    s1, stt, b = host(out["s1"]), host(out["stats"]).reshape(batch.n_heads, batch.n_seqs, 4), host(out["best_ret"])
    for (h, s) in problems:
        a, e = int(batch.cu_seqlens[s]), int(batch.cu_seqlens[s + 1])
        k, r = batch.keys[h, a:e], batch.retained[h, a:e]
        orc = oracle.repair_problem(k, batch.dtype, r, batch.budget[s], tau, w, n_sink, n_recent)
        rows = np.arange(e - a)
        g = {key: host(out[key][h, a:e]) for key in ("best_all", "arg_all", "best_ret", "arg_ret")}
        st = check_scores(g, orc, rows, k, batch.dtype, r, w)
        rr = check_repair(s1[h, a:e], stt[h, s], b[h, a:e], orc, r, tau, n_sink, n_recent)
        res.append((h, s, st, rr))
    return res


def run_repair(batch):
    sp = batch.spec
    kt, rt = to_device(batch.keys, batch.dtype), mask_to_device(batch.retained)
    out = binding.repair(kt, rt, batch.budget, sp.tau, sp.w, sp.n_sink, sp.n_recent, batch.cu_seqlens)
    import torch
    torch.cuda.synchronize()
    return out


def test_tiny_full_parity():
    batch = synth.make_batch(synth.spec("tiny"))
    sp = batch.spec
    out = run_repair(batch)
    res = check_full_problems(batch, out, [(0, 0)], sp.tau, sp.w, sp.n_sink, sp.n_recent)
    print("tiny", res)
    assert res[0][3]["exact"], "tiny: S1 differs from the oracle"


def test_llama1b_8k():
    batch = synth.make_batch(synth.spec("llama1b_8k"))
    sp = batch.spec
    out = run_repair(batch)
    swapped = check_all_problems(batch, out, sp.tau, sp.n_sink, sp.n_recent)
    rng = np.random.default_rng(1)
    agg = check_sampled_rows(batch, out, [(0, 0), (77, 0), (127, 0)], rng, sp.w)
    res = check_full_problems(batch, out, [(5, 0), (100, 0)], sp.tau, sp.w, sp.n_sink, sp.n_recent)
    print("llama1b_8k swapped", swapped, "sampled", agg, "full", [(r[0], r[3]) for r in res])


@pytest.mark.parametrize("frac", synth.QWEN_SWEEP_BUDGETS)
def test_qwen4b_16k_sweep(frac):
    batch = synth.make_batch(synth.spec("qwen4b_16k"), budget_frac=frac, threads=16)
    sp = batch.spec
    kt, rt = to_device(batch.keys, batch.dtype), mask_to_device(batch.retained)
    rng = np.random.default_rng(2)
    for tau in synth.QWEN_SWEEP_TAUS:
        out = binding.repair(kt, rt, batch.budget, tau, sp.w, sp.n_sink, sp.n_recent, batch.cu_seqlens)
        swapped = check_all_problems(batch, out, tau, sp.n_sink, sp.n_recent)
        if tau == synth.QWEN_SWEEP_TAUS[0]:
            agg = check_sampled_rows(batch, out, [(3, 0), (200, 0)], rng, sp.w)
            print("qwen4b_16k", frac, "sampled", agg)
        print("qwen4b_16k", frac, tau, "swapped", swapped)


def test_long_aniso_32k():
    batch = synth.make_batch(synth.spec("long_aniso_32k"), threads=16)
    sp = batch.spec
    out = run_repair(batch)
    swapped = check_all_problems(batch, out, sp.tau, sp.n_sink, sp.n_recent)
    rng = np.random.default_rng(3)
    agg = check_sampled_rows(batch, out, [(0, 0), (131, 0), (287, 0)], rng, sp.w)
    print("long_aniso_32k swapped", swapped, "sampled", agg)


def test_ragged_64x_one_launch():
    batch = synth.make_batch(synth.spec("ragged_64x"), threads=16)
    sp = batch.spec
    out = run_repair(batch)
    swapped = check_all_problems(batch, out, sp.tau, sp.n_sink, sp.n_recent)
    lens = np.diff(batch.cu_seqlens)
    shortest, longest = int(np.argmin(lens)), int(np.argmax(lens))
    probs = [(0, shortest), (287, longest), (100, 5), (9, 40)]
    res = check_full_problems(batch, out, probs, sp.tau, sp.w, sp.n_sink, sp.n_recent)
    print("ragged_64x swapped", swapped, "full", [(r[0], r[1], r[3]) for r in res])

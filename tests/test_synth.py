"""The seeded input generator (shared by the oracle and the HIP path, holds none of the
method's arithmetic) against the workload recipes, and bench.py's single-GPU contract.
CPU only; reduced sequence lengths where the recipe does not depend on them."""
import os
import subprocess
import sys

import numpy as np

from paper_2608_27128_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def cosines(K):
    K = K.astype(np.float64)
    K = K / np.linalg.norm(K, axis=1, keepdims=True)
    return K @ K.T


def test_tiny_recipe():
    """1 x 512 x 64 fp32 i.i.d. keys, 10% planted near-duplicates of an earlier key
    (sigma 0.01), budget 256 with positions 0-3 and the last 32 forced into S0."""
    b = synth.make_batch(synth.spec("tiny"))
    assert b.keys.shape == (1, 512, 64) and b.keys.dtype == np.float32
    r = b.retained[0]
    assert r.sum() == 256 and r[:4].all() and r[-32:].all()
    C = cosines(b.keys[0])
    earlier = np.tril(C, -1)
    # every planted copy has an earlier near-duplicate, nothing else comes close
    assert int((earlier.max(axis=1) > 0.99).sum()) == 51
    off = C[~np.eye(512, dtype=bool)]
    assert float(np.median(np.abs(off))) < 0.15      # i.i.d. keys: cosines ~ N(0, 1/64)


def test_llama_recipe_reduced():
    """bf16 channel-offset keys (per-problem channel mean with sd 2), budget floor(0.5 n),
    4 sinks and the last 64 positions forced."""
    sp = synth.spec("llama1b_8k", n_heads=3, lens=(1024,))
    b = synth.make_batch(sp)
    assert b.keys.shape == (3, 1024, 64) and b.keys.dtype == np.uint16
    assert np.array_equal(b.budget, [512])
    for h in range(3):
        r = b.retained[h]
        assert r.sum() == 512 and r[:4].all() and r[-64:].all()
        K = synth.bf16_to_f32(b.keys[h])
        sd_means = float(K.mean(axis=0).std())
        assert 1.3 < sd_means < 2.7, sd_means
        # 15% planted copies (sigma 0.02 on keys of norm ~17): cosine above 0.999
        assert int((np.tril(cosines(K), -1).max(axis=1) > 0.999).sum()) >= 150


def test_qwen_budgets_nested():
    """The sweep's three retained sets come from one score draw: nested, on identical keys."""
    sp = synth.spec("qwen4b_16k", n_heads=2, lens=(2048,))
    sets, keys = [], None
    for f in synth.QWEN_SWEEP_BUDGETS:
        b = synth.make_batch(sp, budget_frac=f)
        assert np.array_equal(b.budget, [int(np.floor(f * 2048))])
        assert np.all(b.retained.sum(axis=1) == b.budget[0])
        assert np.all(b.retained[:, :4] == 1)
        if keys is None:
            keys = b.keys
        assert np.array_equal(b.keys, keys)
        sets.append(b.retained.astype(bool))
    assert np.all(sets[0] <= sets[1]) and np.all(sets[1] <= sets[2])


def test_long_aniso_recipe_reduced():
    """Budget floor(0.3 n) with 4 sinks and 128 recent positions; four outlier channels of
    magnitude 20 (spread over rotate-half pairs by RoPE) dominate the key norms."""
    sp = synth.spec("long_aniso_32k", n_heads=1, lens=(2048,))
    b = synth.make_batch(sp)
    r = b.retained[0]
    assert r.sum() == 614 and r[:4].all() and r[-128:].all()
    K = synth.bf16_to_f32(b.keys[0]).astype(np.float64)
    norms = np.linalg.norm(K, axis=1)
    # E||k||^2 = 8 * 128 (rank-8 part) + 4 * 20^2 (outliers) + 128 (noise) = 2752
    assert 47.0 < float(np.median(norms)) < 58.0


def test_ragged_recipe():
    sp = synth.spec("ragged_64x")
    assert len(sp.lens) == 64 and min(sp.lens) >= 1024 and max(sp.lens) <= 4096
    assert sp.lens == synth.spec("ragged_64x").lens            # seeded
    small = synth.spec("ragged_64x", n_heads=2, lens=sp.lens[:3])
    b = synth.make_batch(small)
    assert np.array_equal(b.budget, [L // 2 for L in sp.lens[:3]])
    for s in range(3):
        a, e = b.cu_seqlens[s], b.cu_seqlens[s + 1]
        assert np.all(b.retained[:, a:e].sum(axis=1) == sp.lens[s] // 2)
        assert np.all(b.retained[:, a:a + 4] == 1)


def test_generation_is_deterministic_and_thread_independent():
    sp = synth.spec("llama1b_8k", n_heads=4, lens=(300, 0, 77))
    b1 = synth.make_batch(sp, threads=1)
    b2 = synth.make_batch(sp, threads=4)
    assert np.array_equal(b1.keys, b2.keys) and np.array_equal(b1.retained, b2.retained)
    assert np.array_equal(b1.cu_seqlens, [0, 300, 300, 377])


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "exactly one GPU" in r.stderr

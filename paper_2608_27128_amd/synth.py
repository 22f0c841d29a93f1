"""Seeded synthetic KV-cache workloads for the TwinKV redundancy/repair path.

This module produces *inputs only*: post-RoPE-like key tensors, a retained set
S0 chosen by a synthetic wrapped eviction policy, its budget, and the repair
parameters.  It contains none of the method's arithmetic (no normalisation,
no similarity, no twin search, no orphan/donor logic), so both the HIP path
and the CPU oracle can consume the same arrays without sharing method code.

Why synthetic: the paper's measurements use real caches of Qwen3-4B and
Llama-3.2-1B on LongBench / LooGLE / RULER / MMLU-Pro (Sec. 4.1), none of which
is available here.  The recipes below stand in for them with the shapes of
those models (16 layers x 8 KV heads x d=64; 36 layers x 8 KV heads x d=128),
keys as stored in the cache after RoPE (Sec. 3.2, last paragraph), and planted
near-duplicates so that twins exist at controlled rates (the paper reports
37-47% of real tokens having a twin, Sec. 2.2 / Fig. 1b).

Layout of a batch (all numpy, host memory):
  keys       (n_heads, T, d)  uint16 raw bf16 bits, or float32
  retained   (n_heads, T)     uint8 0/1, the wrapped policy's S0
  budget     (n_seqs,)        int64, |S0| of every (head, sequence) problem
  cu_seqlens (n_seqs + 1,)    int64, sequence s owns tokens [cu[s], cu[s+1])
where n_heads counts (layer, KV head) pairs and T = cu_seqlens[-1].

Randomness: every (sequence, head) problem draws from its own PCG64 stream,
seeded by SeedSequence(seed, spawn_key=(config_id, s, h)), in a fixed order
(base keys, planted duplicates, policy scores).  A single problem can be
regenerated on its own (``problem()``) and is identical to the same slice of
the full batch.
"""
from __future__ import annotations

import math
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field, replace
from typing import List, Optional, Sequence, Tuple

import numpy as np

__all__ = [
    "Spec", "Batch", "CONFIGS", "spec", "make_batch", "problem",
    "bf16_bits", "bf16_to_f32",
]


# ----------------------------------------------------------------------------
# bf16 helpers (storage format only)
# ----------------------------------------------------------------------------
def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32/float64 values to bf16 (round-to-nearest-even); return raw uint16 bits."""
    f = np.ascontiguousarray(x, dtype=np.float32)
    u = f.view(np.uint32)
    # finite inputs stay below 2^32 after adding the rounding increment
    rounded = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return rounded.astype(np.uint16)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of raw bf16 bits to float32."""
    return (bits.astype(np.uint32) << 16).view(np.float32)


# ----------------------------------------------------------------------------
# Workload specification
# ----------------------------------------------------------------------------
@dataclass(frozen=True)
class Spec:
    """A seeded synthetic workload.

    key_recipe:
      "iid"     k_t ~ N(0, 1)^d
      "offset"  k_t = mu + N(0, 1)^d with a per-problem channel mean mu ~ N(0, offset_sd^2)^d
      "aniso"   k_t = U z_t + o + eps_t, U in R^{d x rank} N(0,1), z_t ~ N(0, I_rank),
                o = +-outlier_mag on n_outliers seeded channels, eps ~ N(0,1); then
                rotary position embedding (rotate-half pairs (c, c+d/2), theta_c =
                rope_base^(-2c/d), angle pos*theta_c) applied AFTER duplicates are planted.
    dup_recipe:
      "uniform"   floor(dup_frac*n) targets t drawn without replacement from 1..n-1,
                  processed in ascending order: k_t <- k_s + N(0, dup_sigma^2), s ~ U[0, t).
      "clusters"  clusters of cluster_min..cluster_max members: one source position and
                  (size-1) copies at fresh random positions, each copy = source + noise,
                  until floor(dup_frac*n) copies are planted.
    Policy (the wrapped eviction policy that produces S0):
      score_recipe "uniform" U(0,1) or "recency" U(0,1) + recency_weight*pos/n;
      sinks [0, policy_sinks) and the last policy_recent positions get score +inf;
      S0 = top-B by score (ties -> lower index), B = fixed_budget or floor(budget_frac*n).
    Repair parameters: tau, w, n_sink, n_recent (the protected regions used by the repair).
    """
    name: str
    config_id: int
    n_heads: int
    lens: Tuple[int, ...]
    d: int
    dtype: str                      # "bf16" or "f32"
    key_recipe: str
    dup_recipe: str
    dup_frac: float
    dup_sigma: float
    score_recipe: str = "uniform"
    budget_frac: float = 0.5
    fixed_budget: Optional[int] = None
    policy_sinks: int = 4
    policy_recent: int = 0
    tau: float = 0.9
    w: int = 32
    n_sink: int = 4
    n_recent: int = 0
    seed: int = 0
    offset_sd: float = 2.0
    rank: int = 8
    n_outliers: int = 4
    outlier_mag: float = 20.0
    rope_base: float = 1.0e6
    cluster_min: int = 2
    cluster_max: int = 8
    recency_weight: float = 0.5

    @property
    def n_seqs(self) -> int:
        return len(self.lens)

    @property
    def total_tokens(self) -> int:
        return int(sum(self.lens))

    def budget_of(self, n: int) -> int:
        if self.fixed_budget is not None:
            return int(self.fixed_budget)
        return int(math.floor(self.budget_frac * n))


@dataclass
class Batch:
    spec: Spec
    keys: np.ndarray
    retained: np.ndarray
    budget: np.ndarray
    cu_seqlens: np.ndarray

    @property
    def dtype(self) -> str:
        return self.spec.dtype

    @property
    def n_heads(self) -> int:
        return self.keys.shape[0]

    @property
    def d(self) -> int:
        return self.keys.shape[2]

    @property
    def n_seqs(self) -> int:
        return len(self.cu_seqlens) - 1

    def seq(self, h: int, s: int):
        """(keys, retained) views of problem (head h, sequence s)."""
        a, b = int(self.cu_seqlens[s]), int(self.cu_seqlens[s + 1])
        return self.keys[h, a:b], self.retained[h, a:b]


def _ragged_lens(seed: int, n_seqs: int, lo: int, hi: int) -> Tuple[int, ...]:
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=(99, 0))))
    return tuple(int(x) for x in g.integers(lo, hi + 1, size=n_seqs))


def _configs() -> dict:
    c = {}
    # Tiny: 1 layer x 1 KV head, N=512, d=64, fp32 i.i.d. N(0,1); 10% near-duplicates
    # (sigma 0.01); B=256 from uniform scores with sinks 0-3 and the last 32 forced.
    c["tiny"] = Spec(name="tiny", config_id=0, n_heads=1, lens=(512,), d=64, dtype="f32",
                     key_recipe="iid", dup_recipe="uniform", dup_frac=0.10, dup_sigma=0.01,
                     fixed_budget=256, policy_sinks=4, policy_recent=32,
                     tau=0.9, w=32, n_sink=4, n_recent=32)
    # Llama-3.2-1B-shaped cache: 16 layers x 8 KV heads, d=64, N=8192, bf16; channel-offset
    # keys; 15% near-duplicates (sigma 0.02); B=floor(0.5N) with 4 sinks + 64 recent.
    c["llama1b_8k"] = Spec(name="llama1b_8k", config_id=1, n_heads=16 * 8, lens=(8192,), d=64,
                           dtype="bf16", key_recipe="offset", dup_recipe="uniform",
                           dup_frac=0.15, dup_sigma=0.02, budget_frac=0.5,
                           policy_sinks=4, policy_recent=64, tau=0.9, w=32, n_sink=4, n_recent=64)
    # Qwen3-4B-shaped cache: 36 x 8, d=128, N=16384, keys as above; budgets 0.3/0.5/0.7 of N
    # from recency-favouring scores (U + 0.5 pos/N) plus 4 sinks; tau sweep 0.85/0.9/0.95.
    c["qwen4b_16k"] = Spec(name="qwen4b_16k", config_id=2, n_heads=36 * 8, lens=(16384,), d=128,
                           dtype="bf16", key_recipe="offset", dup_recipe="uniform",
                           dup_frac=0.15, dup_sigma=0.02, score_recipe="recency",
                           budget_frac=0.5, policy_sinks=4, policy_recent=0,
                           tau=0.9, w=32, n_sink=4, n_recent=0)
    # Long, anisotropic: 36 x 8, d=128, N=32768, bf16; rank-8 shared component + 4 outlier
    # channels of magnitude 20 + N(0,1), RoPE base 1e6; 20% near-duplicates in clusters of
    # 2-8; B=floor(0.3N) from uniform scores + 4 sinks + 128 recent.
    c["long_aniso_32k"] = Spec(name="long_aniso_32k", config_id=3, n_heads=36 * 8, lens=(32768,),
                               d=128, dtype="bf16", key_recipe="aniso", dup_recipe="clusters",
                               dup_frac=0.20, dup_sigma=0.02, budget_frac=0.3,
                               policy_sinks=4, policy_recent=128, tau=0.9, w=32,
                               n_sink=4, n_recent=128)
    # Ragged short-context batch: 64 sequences, len ~ U[1024, 4096], 36 x 8, d=128, bf16,
    # channel-offset keys with 5% near-duplicates; per-sequence B=floor(0.5 len) + 4 sinks.
    c["ragged_64x"] = Spec(name="ragged_64x", config_id=4, n_heads=36 * 8,
                           lens=_ragged_lens(0, 64, 1024, 4096), d=128, dtype="bf16",
                           key_recipe="offset", dup_recipe="uniform", dup_frac=0.05,
                           dup_sigma=0.02, budget_frac=0.5, policy_sinks=4, policy_recent=0,
                           tau=0.9, w=32, n_sink=4, n_recent=0)
    return c


CONFIGS = _configs()

#: The retained fractions and thresholds swept by the Qwen3-4B-shaped workload.
QWEN_SWEEP_BUDGETS = (0.3, 0.5, 0.7)
QWEN_SWEEP_TAUS = (0.85, 0.9, 0.95)


def spec(name: str, **overrides) -> Spec:
    """A named workload, optionally with fields replaced (e.g. smaller lens for tests)."""
    base = CONFIGS[name]
    return replace(base, **overrides) if overrides else base


# ----------------------------------------------------------------------------
# Per-problem generation
# ----------------------------------------------------------------------------
def _rng(sp: Spec, s: int, h: int) -> np.random.Generator:
    ss = np.random.SeedSequence(sp.seed, spawn_key=(sp.config_id, s, h))
    return np.random.Generator(np.random.PCG64(ss))


def _base_keys(sp: Spec, g: np.random.Generator, n: int) -> np.ndarray:
    d = sp.d
    f32 = np.float32
    if sp.key_recipe == "iid":
        return g.standard_normal((n, d), dtype=f32)
    if sp.key_recipe == "offset":
        mu = g.normal(0.0, sp.offset_sd, size=d).astype(f32)
        K = g.standard_normal((n, d), dtype=f32)
        K += mu[None, :]
        return K
    if sp.key_recipe == "aniso":
        U = g.standard_normal((d, sp.rank), dtype=f32)
        z = g.standard_normal((n, sp.rank), dtype=f32)
        chans = g.choice(d, size=sp.n_outliers, replace=False)
        signs = np.where(g.random(sp.n_outliers) < 0.5, -1.0, 1.0)
        o = np.zeros(d, dtype=f32)
        o[chans] = signs * sp.outlier_mag
        K = z @ U.T
        K += o[None, :]
        K += g.standard_normal((n, d), dtype=f32)
        return K
    raise ValueError(f"unknown key recipe {sp.key_recipe!r}")


def _resolve_copies(K: np.ndarray, tgt: np.ndarray, src: np.ndarray, noise: np.ndarray) -> None:
    """Apply k[tgt] <- k[src] + noise in ascending target order (src < tgt).

    A source may itself be an earlier target, so the assignment is a chain; it is
    resolved by repeating the simultaneous update until every chain has propagated
    (the depth of the longest chain), which equals the sequential ascending-order result.
    """
    if len(tgt) == 0:
        return
    n = K.shape[0]
    depth = np.zeros(n, dtype=np.int64)
    is_t = np.zeros(n, dtype=bool)
    is_t[tgt] = True
    # chain depth: depth[t] = 1 + depth[src] (src processed first because src < t)
    order = np.argsort(tgt)
    tgt, src, noise = tgt[order], src[order], noise[order]
    while True:
        nd = depth.copy()
        nd[tgt] = 1 + depth[src]
        if np.array_equal(nd, depth):
            break
        depth = nd
    for _ in range(int(depth.max())):
        K[tgt] = K[src] + noise
    # the fixed point satisfies the definition exactly
    assert np.array_equal(K[tgt], K[src] + noise)


def _plant(sp: Spec, g: np.random.Generator, K: np.ndarray) -> None:
    n, d = K.shape
    n_copies = int(math.floor(sp.dup_frac * n))
    if n_copies == 0 or n < 2:
        return
    if sp.dup_recipe == "uniform":
        tgt = np.sort(g.choice(np.arange(1, n), size=min(n_copies, n - 1), replace=False))
        src = np.floor(g.random(len(tgt)) * tgt).astype(np.int64)   # uniform in [0, t)
        noise = (sp.dup_sigma * g.standard_normal((len(tgt), d), dtype=np.float32))
        _resolve_copies(K, tgt, src, noise)
        return
    if sp.dup_recipe == "clusters":
        # positions are consumed without replacement: each cluster takes `size` fresh
        # positions; the first is the source, the rest become its copies.
        perm = g.permutation(n)
        used = 0
        planted = 0
        tg, sr = [], []
        while planted < n_copies and used + 2 <= n:
            size = int(g.integers(sp.cluster_min, sp.cluster_max + 1))
            size = min(size, n_copies - planted + 1, n - used)
            if size < 2:
                break
            members = perm[used:used + size]
            used += size
            s0 = int(members[0])
            for t in members[1:]:
                tg.append(int(t))
                sr.append(s0)
            planted += size - 1
        tgt = np.asarray(tg, dtype=np.int64)
        src = np.asarray(sr, dtype=np.int64)
        noise = (sp.dup_sigma * g.standard_normal((len(tgt), d), dtype=np.float32))
        # sources are never targets here, so a single simultaneous update is exact
        K[tgt] = K[src] + noise
        return
    raise ValueError(f"unknown duplicate recipe {sp.dup_recipe!r}")


def _rope(sp: Spec, K: np.ndarray) -> np.ndarray:
    n, d = K.shape
    half = d // 2
    c = np.arange(half, dtype=np.float64)
    theta = sp.rope_base ** (-2.0 * c / d)
    ang = np.arange(n, dtype=np.float64)[:, None] * theta[None, :]
    cs, sn = np.cos(ang).astype(np.float32), np.sin(ang).astype(np.float32)
    x, y = K[:, :half], K[:, half:]
    return np.concatenate([x * cs - y * sn, x * sn + y * cs], axis=1)


def _policy(sp: Spec, g: np.random.Generator, n: int) -> np.ndarray:
    """Synthetic wrapped eviction policy: top-B of seeded scores with protected regions forced."""
    u = g.random(n)
    if sp.score_recipe == "uniform":
        score = u
    elif sp.score_recipe == "recency":
        score = u + sp.recency_weight * np.arange(n) / n
    else:
        raise ValueError(f"unknown score recipe {sp.score_recipe!r}")
    score = score.copy()
    score[: min(sp.policy_sinks, n)] = np.inf
    if sp.policy_recent > 0:
        score[max(0, n - sp.policy_recent):] = np.inf
    B = sp.budget_of(n)
    order = np.argsort(-score, kind="stable")          # ties -> lower index first
    keep = np.zeros(n, dtype=np.uint8)
    keep[order[:B]] = 1
    return keep


def problem(sp: Spec, s: int, h: int, budget_frac: Optional[float] = None):
    """Keys (n, d) [uint16 bf16 bits or float32] and S0 (n,) uint8 of problem (seq s, head h).

    ``budget_frac`` overrides the spec's retained fraction while keeping the same score
    draw, so different budgets give nested retained sets over identical keys.
    """
    n = int(sp.lens[s])
    g = _rng(sp, s, h)
    K = _base_keys(sp, g, n)
    _plant(sp, g, K)
    if sp.key_recipe == "aniso":
        K = _rope(sp, K)
    sp_pol = sp if budget_frac is None else replace(sp, budget_frac=budget_frac, fixed_budget=None)
    keep = _policy(sp_pol, g, n)
    if sp.dtype == "bf16":
        keys = bf16_bits(K)
    elif sp.dtype == "f32":
        keys = K.astype(np.float32)
    else:
        raise ValueError(f"unknown dtype {sp.dtype!r}")
    return keys, keep


def make_batch(sp: Spec, budget_frac: Optional[float] = None, threads: int = 8) -> Batch:
    """Generate the whole (n_heads, T, d) batch; problems are generated in parallel."""
    T = sp.total_tokens
    cu = np.zeros(sp.n_seqs + 1, dtype=np.int64)
    cu[1:] = np.cumsum(sp.lens)
    kdt = np.uint16 if sp.dtype == "bf16" else np.float32
    keys = np.empty((sp.n_heads, T, sp.d), dtype=kdt)
    ret = np.empty((sp.n_heads, T), dtype=np.uint8)

    def work(job):
        s, h = job
        k, r = problem(sp, s, h, budget_frac=budget_frac)
        a, b = cu[s], cu[s + 1]
        keys[h, a:b] = k
        ret[h, a:b] = r

    jobs = [(s, h) for s in range(sp.n_seqs) for h in range(sp.n_heads)]
    if threads > 1 and len(jobs) > 1:
        with ThreadPoolExecutor(max_workers=threads) as ex:
            list(ex.map(work, jobs))
    else:
        for j in jobs:
            work(j)
    sp_b = sp if budget_frac is None else replace(sp, budget_frac=budget_frac, fixed_budget=None)
    budget = np.array([sp_b.budget_of(n) for n in sp.lens], dtype=np.int64)
    return Batch(spec=sp_b, keys=keys, retained=ret, budget=budget, cu_seqlens=cu)

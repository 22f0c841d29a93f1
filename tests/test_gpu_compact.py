"""KV compaction (Sec. 3.1): HIP path vs the CPU oracle through the C ABI.

A byte copy, so the bar is bit-exact: the compacted keys and values are compared as raw
bytes with the oracle's, and the positions and per-problem stats exactly.  Value vectors
are the key bytes XOR a fixed pattern (any bit pattern is a valid row to copy), so a kernel
that mixes up keys and values, heads or rows fails even with a single head."""
import numpy as np
import pytest

import oracle
from gpu_util import host, mask_to_device, to_device
from paper_2608_27128_amd import binding, synth

pytestmark = pytest.mark.gpu


def values_of(keys_np, dtype):
    """Seeded stand-in for value vectors: the key bits XOR a fixed pattern."""
    if dtype == "bf16":
        return keys_np ^ np.uint16(0x5A5A)
    return (keys_np.view(np.uint32) ^ np.uint32(0x5A5A5A5A)).view(np.float32)


def as_bytes(x):
    return np.ascontiguousarray(x).view(np.uint8)


def raw(t):
    """Host copy of a GPU tensor's elements as plain bits (numpy has no bf16)."""
    import torch
    return host(t.view(torch.int16) if t.dtype == torch.bfloat16 else t)


def check_against_oracle(keys_np, vals_np, dtype, mask, cu, cap, out):
    o = oracle.compact(keys_np, vals_np, mask, cu, cap)
    np.testing.assert_array_equal(host(out["stats"]), o["stats"])
    np.testing.assert_array_equal(host(out["pos"]), o["pos"])
    assert np.array_equal(as_bytes(raw(out["keys"])), as_bytes(o["keys"])), "compacted keys differ"
    if vals_np is not None:
        assert np.array_equal(as_bytes(raw(out["values"])), as_bytes(o["values"])), \
            "compacted values differ"
    return o


def small_batch(H, lens, d, dtype, seed):
    sp = synth.Spec(name="compact", config_id=90 + seed % 7, n_heads=H, lens=tuple(lens), d=d,
                    dtype=dtype, key_recipe="offset", dup_recipe="uniform", dup_frac=0.1,
                    dup_sigma=0.02, budget_frac=0.4, policy_sinks=4, policy_recent=8, tau=0.9,
                    w=32, n_sink=4, n_recent=8, seed=seed)
    return synth.make_batch(sp)


CASES = [
    # (heads, lens, d, dtype, capacity mode, with values)
    (2, [700], 64, "bf16", "budget", True),
    (3, [2047, 2048, 2049], 128, "bf16", "budget", True),         # chunk boundaries
    (2, [4100, 1, 0, 33], 128, "bf16", "slack", True),             # ragged, empty, slack rows
    (1, [900], 64, "f32", "budget", True),
    (2, [5000], 128, "f32", "slack", False),                       # keys only, 512-byte rows
    (4, [300, 2500], 64, "bf16", "tight", True),                   # every problem overflows
    (9, [1200, 64], 128, "bf16", "random", True),                  # random masks and rows
]


@pytest.mark.parametrize("H,lens,d,dtype,mode,with_values", CASES)
def test_compact_vs_oracle(H, lens, d, dtype, mode, with_values):
    seed = (H * 31 + sum(lens) + d) % 1009
    batch = small_batch(H, lens, d, dtype, seed)
    cu = batch.cu_seqlens
    mask = batch.retained.copy()
    budget = np.asarray(batch.budget, dtype=np.int64)
    lens_a = np.diff(cu)
    rng = np.random.default_rng(seed)
    if mode == "budget":
        cap = budget
    elif mode == "slack":
        cap = np.minimum(lens_a, budget + 7)
    elif mode == "tight":
        cap = np.maximum(budget - 1, 0)
    else:
        mask = (rng.random(mask.shape) < 0.3).astype(np.uint8)
        cap = np.array([int(rng.integers(0, L + 1)) for L in lens_a], dtype=np.int64)
    vals = values_of(batch.keys, dtype) if with_values else None
    out = binding.compact(to_device(batch.keys, dtype), mask_to_device(mask), cap,
                          values=None if vals is None else to_device(vals, dtype), cu_seqlens=cu)
    o = check_against_oracle(batch.keys, vals, dtype, mask, cu, cap, out)
    st = o["stats"]
    print("compact", H, lens, d, dtype, mode, "kept", int(st[:, 0].sum()), "overflow",
          int(st[:, 2].sum()))
    if mode == "tight":
        assert np.all(st[:, 2] == (st[:, 0] > st[:, 1]))


def test_compact_strided_inputs():
    """Keys and values as strided views (token stride 2d, separate head strides)."""
    import torch
    batch = small_batch(3, [1500, 700], 64, "bf16", 5)
    H, T, d = batch.keys.shape
    big = np.zeros((H, T, 2 * d), dtype=np.uint16)
    big[:, :, :d] = batch.keys
    vals = values_of(batch.keys, "bf16")
    vbig = np.zeros((H + 1, T, d), dtype=np.uint16)
    vbig[1:] = vals
    kt = to_device(big, "bf16")[:, :, :d]
    vt = to_device(vbig, "bf16")[1:]
    assert kt.stride(1) == 2 * d and vt.stride(0) == T * d
    out = binding.compact(kt, mask_to_device(batch.retained), batch.budget, values=vt,
                          cu_seqlens=batch.cu_seqlens)
    check_against_oracle(batch.keys, vals, "bf16", batch.retained, batch.cu_seqlens,
                         np.asarray(batch.budget), out)
    torch.cuda.synchronize()


def test_compact_after_repair():
    """The pipeline the paper implies: repair S0 into S1, then keep the S1 rows; each problem
    keeps exactly its budget (|S1| = |S0| = K)."""
    batch = small_batch(4, [3000, 900], 128, "bf16", 11)
    sp = batch.spec
    kt = to_device(batch.keys, "bf16")
    rep = binding.repair(kt, mask_to_device(batch.retained), batch.budget, sp.tau, sp.w,
                         sp.n_sink, sp.n_recent, batch.cu_seqlens)
    s1 = host(rep["s1"])
    vals = values_of(batch.keys, "bf16")
    out = binding.compact(kt, rep["s1"], batch.budget, values=to_device(vals, "bf16"),
                          cu_seqlens=batch.cu_seqlens)
    o = check_against_oracle(batch.keys, vals, "bf16", s1, batch.cu_seqlens,
                             np.asarray(batch.budget), out)
    bud = np.tile(np.asarray(batch.budget), batch.n_heads)
    np.testing.assert_array_equal(o["stats"][:, 0], bud)
    assert np.all(o["stats"][:, 2] == 0)


def test_compact_reuses_outputs():
    """Two calls into the same buffers: the second, with fewer kept rows, leaves no stale rows."""
    batch = small_batch(2, [2100], 64, "bf16", 3)
    kt = to_device(batch.keys, "bf16")
    cap = np.asarray(batch.budget)
    out = binding.compact(kt, mask_to_device(batch.retained), cap, cu_seqlens=batch.cu_seqlens)
    m2 = batch.retained.copy()
    m2[:, ::3] = 0
    out2 = binding.compact(kt, mask_to_device(m2), cap, cu_seqlens=batch.cu_seqlens, outputs=out)
    check_against_oracle(batch.keys, None, "bf16", m2, batch.cu_seqlens, cap, out2)


def test_compact_full_long_aniso_32k():
    """The 36x8 x 32768 x 128 bf16 cache at its S0 (9830 rows per problem), keys and values,
    in the launch configuration the benchmark times: every problem against the oracle."""
    batch = synth.make_batch(synth.spec("long_aniso_32k"), threads=16)
    vals = values_of(batch.keys, "bf16")
    cap = np.asarray(batch.budget)
    out = binding.compact(to_device(batch.keys, "bf16"), mask_to_device(batch.retained), cap,
                          values=to_device(vals, "bf16"), cu_seqlens=batch.cu_seqlens)
    o = check_against_oracle(batch.keys, vals, "bf16", batch.retained, batch.cu_seqlens, cap, out)
    assert np.all(o["stats"][:, 0] == cap[0]) and np.all(o["stats"][:, 2] == 0)

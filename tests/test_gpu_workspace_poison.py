"""Results do not depend on what the caller's workspace held before the call.

The similarity sweep pads column groups with slots whose keys are never written (their
inverse norms are 0 and their chunks are dropped by the kernel's masks).  A mask that lets
such a chunk through is invisible on a zeroed workspace (its candidates score 0) but not on
one full of 0xFF bytes, whose bf16 keys are NaN.  Every path runs once on a zeroed and once
on a poisoned workspace, and the results must agree bit for bit.
"""
import numpy as np
import pytest

from gpu_util import host, mask_to_device, to_device
from paper_2608_27128_amd import binding, synth

pytestmark = pytest.mark.gpu

CASES = [
    # (heads, lengths, d, dtype, w): ragged lengths put padding chunks into the last S0 tile
    (3, [1500, 700, 0, 33], 128, "bf16", 32),
    (9, [2100, 389], 128, "bf16", 32),
    (2, [1000, 77], 64, "bf16", 16),
    (2, [640, 300], 64, "f32", 8),
    (2, [513, 260], 128, "f32", 32),
]


def spec_of(H, lens, d, dtype, w, seed):
    return synth.Spec(name="poison", config_id=90 + seed, n_heads=H, lens=tuple(lens), d=d,
                      dtype=dtype, key_recipe="offset", dup_recipe="uniform", dup_frac=0.15,
                      dup_sigma=0.02, budget_frac=0.3, policy_sinks=4, policy_recent=0,
                      tau=0.9, w=w, n_sink=4, n_recent=0, seed=seed)


def workspaces(nbytes):
    import torch
    zero = torch.zeros((nbytes,), dtype=torch.uint8, device="cuda")
    poison = torch.full((nbytes,), 0xFF, dtype=torch.uint8, device="cuda")
    return zero, poison


def same(a: dict, b: dict, keys):
    for k in keys:
        x, y = host(a[k]), host(b[k])
        assert x.shape == y.shape, k
        assert np.array_equal(x.view(np.uint8), y.view(np.uint8)), k


@pytest.mark.parametrize("H,lens,d,dtype,w", CASES)
def test_repair_and_scores_ignore_workspace_contents(H, lens, d, dtype, w):
    sp = spec_of(H, lens, d, dtype, w, seed=H + d + w)
    batch = synth.make_batch(sp, threads=16)
    cu = batch.cu_seqlens
    kt = to_device(batch.keys, dtype)
    ret = mask_to_device(batch.retained)
    dt = 0 if dtype == "bf16" else 1
    for want_all in (True, False):
        zero, poison = workspaces(binding.workspace_bytes(binding.OP_REPAIR, dt, d, H, cu))
        r0 = binding.repair(kt, ret, batch.budget, sp.tau, w, sp.n_sink, sp.n_recent, cu,
                            want_all=want_all, workspace=zero)
        r1 = binding.repair(kt, ret, batch.budget, sp.tau, w, sp.n_sink, sp.n_recent, cu,
                            want_all=want_all, workspace=poison)
        keys = ["s1", "stats", "best_ret", "arg_ret"] + (["best_all", "arg_all"] if want_all else [])
        same(r0, r1, keys)
        vals = host(r0["best_ret"])
        assert np.isfinite(vals).all()
        assert (vals >= -1.0 - 1e-6).all() and (vals <= 1.0 + 1e-4).all()
    zero, poison = workspaces(binding.workspace_bytes(binding.OP_NN_SCORES, dt, d, H, cu))
    n0 = binding.nn_scores(kt, ret, w, cu, workspace=zero)
    n1 = binding.nn_scores(kt, ret, w, cu, workspace=poison)
    same(n0, n1, ["best_all", "arg_all", "best_ret", "arg_ret"])
    zero, poison = workspaces(binding.workspace_bytes(binding.OP_TWIN_COUNTS, dt, d, H, cu))
    c0 = binding.twin_counts(kt, sp.tau, w, cu, workspace=zero)
    c1 = binding.twin_counts(kt, sp.tau, w, cu, workspace=poison)
    same(c0, c1, ["counts"])


def test_workspace_on_another_device_or_strided_is_refused():
    """A workspace the kernels could not address as one device buffer (host memory, a strided
    view) is refused before the call; one given as wider elements counts by bytes."""
    import torch
    batch = synth.make_batch(spec_of(2, [300, 41], 128, "bf16", 32, 7))
    sp = batch.spec
    kt, ret = to_device(batch.keys, "bf16"), mask_to_device(batch.retained)
    cu = batch.cu_seqlens
    nbytes = binding.workspace_bytes(binding.OP_REPAIR, 0, 128, 2, cu)
    args = (kt, ret, batch.budget, sp.tau, sp.w, sp.n_sink, sp.n_recent, cu)
    with pytest.raises(ValueError, match="workspace"):
        binding.repair(*args, workspace=torch.zeros((nbytes,), dtype=torch.uint8))
    with pytest.raises(ValueError, match="workspace"):
        binding.repair(*args, workspace=torch.zeros((2 * nbytes,), dtype=torch.uint8,
                                                    device="cuda")[::2])
    ref = binding.repair(*args)
    wide = torch.full(((nbytes + 3) // 4,), -1, dtype=torch.int32, device="cuda")
    got = binding.repair(*args, workspace=wide)
    same(ref, got, ["s1", "stats", "best_ret", "arg_ret", "best_all", "arg_all"])


@pytest.mark.parametrize("H,lens,d,dtype,w", CASES)
def test_levels_ignore_workspace_contents(H, lens, d, dtype, w):
    """The nested-sets call (one key preparation for all level groups, each group's column
    list in its own workspace slice) on a zeroed and on a poisoned workspace."""
    import torch
    batch = synth.make_batch(spec_of(H, lens, d, dtype, w, 5))
    g = np.random.default_rng(5)
    level = g.integers(0, 5, batch.retained.shape).astype(np.uint8)   # 4 = above n_levels
    kt, cu = to_device(batch.keys, dtype), batch.cu_seqlens
    lv = torch.from_numpy(level).cuda()
    dt = 0 if dtype == "bf16" else 1
    for want_all in (False, True):
        nbytes = binding.levels_workspace_bytes(dt, d, H, cu, 3, want_all)
        zero, poison = workspaces(nbytes)
        a = binding.nn_scores_levels(kt, lv, 3, w, cu, want_all=want_all, workspace=zero)
        b = binding.nn_scores_levels(kt, lv, 3, w, cu, want_all=want_all, workspace=poison)
        same(a, b, [k for k in a if k != "status"] + ["status"])
        vals = host(a["best_lvl"])
        assert np.isfinite(vals).all()


def test_concurrent_calls_on_two_streams():
    """Calls with different workspaces may overlap (nothing else is shared between calls):
    two batches repaired at the same time on two streams give what they give one after the
    other, bit for bit."""
    import torch
    b1 = synth.make_batch(spec_of(9, [2100, 389], 128, "bf16", 32, 21))
    b2 = synth.make_batch(spec_of(3, [1500, 700, 0, 33], 128, "bf16", 32, 22))
    args = []
    for b in (b1, b2):
        sp = b.spec
        args.append((to_device(b.keys, "bf16"), mask_to_device(b.retained), b.budget, sp.tau,
                     sp.w, sp.n_sink, sp.n_recent, b.cu_seqlens))
    ref = [binding.repair(*a) for a in args]
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for s in streams:
        s.wait_stream(torch.cuda.current_stream())
    got = [None, None]
    for rep in range(3):
        for i, (s, a) in enumerate(zip(streams, args)):
            with torch.cuda.stream(s):
                got[i] = binding.repair(*a)
        torch.cuda.synchronize()
        for r, g in zip(ref, got):
            same(r, g, ["s1", "stats", "best_ret", "arg_ret", "best_all", "arg_all"])

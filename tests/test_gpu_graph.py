"""The repair call captured into a HIP graph (through torch.cuda.graph): every launch of the
call carries its host tables in kernel arguments, so a replay reads nothing from host memory
that the call has freed.  The graph is replayed several times, with the program's own eager
work and synchronisations between the replays and new keys copied into the captured input
buffers, and every replay is compared with an eager call on the same inputs."""
import numpy as np
import pytest

from gpu_util import host, mask_to_device, to_device
from paper_2608_27128_amd import binding, synth

pytestmark = pytest.mark.gpu


def _batch(seed, lens):
    sp = synth.Spec(name="graph", config_id=140 + seed, n_heads=3, lens=tuple(lens), d=128,
                    dtype="bf16", key_recipe="offset", dup_recipe="uniform", dup_frac=0.2,
                    dup_sigma=0.02, budget_frac=0.5, policy_sinks=2, policy_recent=3, tau=0.9,
                    w=32, n_sink=2, n_recent=3, seed=seed)
    return synth.make_batch(sp)


def test_repair_graph_replays_match_eager():
    import torch
    lens = [900, 37, 1500]
    b0 = _batch(1, lens)
    keys = to_device(b0.keys, "bf16")
    ret = mask_to_device(b0.retained)
    ws = torch.empty((binding.workspace_bytes(binding.OP_REPAIR, 0, 128, 3, b0.cu_seqlens),),
                     dtype=torch.uint8, device="cuda")
    # warm-up on a side stream, as torch asks before capture
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        out = binding.repair(keys, ret, b0.budget, 0.9, 32, 2, 3, b0.cu_seqlens, workspace=ws)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        out = binding.repair(keys, ret, b0.budget, 0.9, 32, 2, 3, b0.cu_seqlens, workspace=ws,
                             outputs=out)
    for rep, seed in enumerate([1, 2, 3, 2]):
        bb = _batch(seed, lens)
        keys.copy_(to_device(bb.keys, "bf16"))
        # the budget is fixed by the capture: keep S0 of the first batch
        g.replay()
        torch.cuda.synchronize()
        got = {k: host(v).copy() for k, v in out.items()}
        # eager work between replays, on fresh buffers and its own workspace
        ref = binding.repair(to_device(bb.keys, "bf16"), mask_to_device(b0.retained), b0.budget,
                             0.9, 32, 2, 3, b0.cu_seqlens)
        torch.cuda.synchronize()
        for k in ("s1", "stats", "best_ret", "arg_ret", "best_all", "arg_all"):
            assert np.array_equal(got[k], host(ref[k])), (rep, k)

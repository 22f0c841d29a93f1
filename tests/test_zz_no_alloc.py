"""twinkv_repair_from_scores_noalloc (no workspace; the sequence table in the library's static
scratch) against twinkv_repair_from_scores, both through the C ABI, on two calls in a row
with the second batch smaller than the first (the static buffer keeps the first call's
table), then a batch at the sequence limit.  Integer outputs: bit for bit."""
import ctypes

import numpy as np
import pytest

from gpu_util import host, mask_to_device
from paper_2608_27128_amd import binding

pytestmark = pytest.mark.gpu


def _i64(v):
    v = [int(x) for x in v]
    return (ctypes.c_int64 * len(v))(*v)


def _case(seed, H, lens):
    g = np.random.default_rng(seed)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    T = int(cu[-1])
    b = (np.round(g.uniform(-1, 1, (H, T)) * 64) / 64).astype(np.float32)  # many ties
    b[g.random((H, T)) < 0.02] = -1.0
    s0 = np.zeros((H, T), np.uint8)
    budget = []
    for s, n in enumerate(lens):
        B = n // 2
        budget.append(B)
        for h in range(H):
            s0[h, cu[s] + g.permutation(n)[:B]] = 1
    return b, s0, cu, budget


def _both(b, s0, cu, budget, tau=0.5, n_sink=3, n_recent=5):
    import torch
    L = binding.lib()
    H, T = b.shape
    n_seqs = len(cu) - 1
    bt, rt = torch.from_numpy(b).cuda(), mask_to_device(s0)
    stream = torch.cuda.current_stream().cuda_stream
    # the existing entry point, with its workspace
    s1_ref = torch.empty((H, T), dtype=torch.uint8, device="cuda")
    st_ref = torch.empty((H * n_seqs, 4), dtype=torch.int32, device="cuda")
    nbytes = binding.workspace_bytes(binding.OP_REPAIR_FROM_SCORES, 0, 64, H, cu)
    ws = torch.empty((nbytes,), dtype=torch.uint8, device="cuda")
    rc = L.twinkv_repair_from_scores(bt.data_ptr(), rt.data_ptr(), s1_ref.data_ptr(), H, n_seqs,
                                     _i64(cu), _i64(budget), tau, n_sink, n_recent,
                                     st_ref.data_ptr(), ws.data_ptr(), nbytes, stream)
    assert rc == 0
    # the variant without allocation: outputs only
    s1 = torch.full((H, T), 7, dtype=torch.uint8, device="cuda")
    st = torch.full((H * n_seqs, 4), -7, dtype=torch.int32, device="cuda")
    rc = L.twinkv_repair_from_scores_noalloc(bt.data_ptr(), rt.data_ptr(), s1.data_ptr(), H,
                                             n_seqs, _i64(cu), _i64(budget), tau, n_sink,
                                             n_recent, st.data_ptr(), stream)
    assert rc == 0, binding.status_string(rc)
    torch.cuda.synchronize()
    assert np.array_equal(host(s1), host(s1_ref))
    assert np.array_equal(host(st), host(st_ref))
    assert np.all(host(st)[:, 3] == 0)
    return host(st)


def test_noalloc_matches_workspace_entry_point_twice():
    # first call: 7 sequences (one past 4096 tokens), then a smaller batch of 3 sequences
    b, s0, cu, bud = _case(5, 4, [5000, 17, 300, 1024, 0, 2048, 999])
    st1 = _both(b, s0, cu, bud)
    assert st1[:, 2].sum() > 0                       # swaps happened
    b, s0, cu, bud = _case(6, 2, [700, 3, 64])
    _both(b, s0, cu, bud)


def test_noalloc_at_sequence_limit():
    n = binding.NOALLOC_MAX_SEQS
    g = np.random.default_rng(9)
    lens = [int(x) for x in g.integers(0, 40, size=n)]
    b, s0, cu, bud = _case(10, 2, lens)
    _both(b, s0, cu, bud)
    # one sequence more is refused before anything is enqueued
    import torch
    L = binding.lib()
    cu2 = np.concatenate([cu, [cu[-1]]])
    bt, rt = torch.from_numpy(b).cuda(), mask_to_device(s0)
    s1 = torch.empty_like(rt)
    st = torch.empty((2 * (n + 1), 4), dtype=torch.int32, device="cuda")
    rc = L.twinkv_repair_from_scores_noalloc(bt.data_ptr(), rt.data_ptr(), s1.data_ptr(), 2, n + 1,
                                             _i64(cu2), _i64(bud + [0]), 0.5, 3, 5, st.data_ptr(),
                                             torch.cuda.current_stream().cuda_stream)
    assert rc == 6

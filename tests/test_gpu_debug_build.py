"""The LDS-race check: libtwinkv_debug.so (built with -DTWINKV_DEBUG: the similarity kernel
poisons each LDS stage once every wave has swept it, behind extra barriers, and the repair
kernel poisons its LDS copy before filling it) must give exactly the product library's
results.  A read of LDS outside the lifetime of what was written there would see the poison.
Both libraries are called through the C ABI on the same inputs."""
import ctypes
import os

import numpy as np
import pytest

from gpu_util import host, mask_to_device, to_device
from paper_2608_27128_amd import binding, build, synth

pytestmark = pytest.mark.gpu


def _debug_lib():
    if not os.path.exists(build.DEBUG_LIB):
        raise RuntimeError(f"{build.DEBUG_LIB} is missing: build with `python -m paper_2608_27128_amd.build`")
    L = ctypes.CDLL(build.DEBUG_LIB)
    for name, (res, args) in binding.SIGNATURES.items():
        f = getattr(L, name)
        f.restype, f.argtypes = res, args
    return L


def _run(L, kt, rt, batch, dt, tau=0.9, w=32):
    import torch
    H, T, d = kt.shape
    n_seqs = len(batch.cu_seqlens) - 1
    cu, bud = binding._i64_array(batch.cu_seqlens), binding._i64_array(batch.budget)
    out = {k: torch.full((H, T), -7, dtype=tp, device="cuda") for k, tp in
           (("s1", torch.uint8), ("best_all", torch.float32), ("arg_all", torch.int32),
            ("best_ret", torch.float32), ("arg_ret", torch.int32), ("counts", torch.int32))}
    out["stats"] = torch.zeros((H * n_seqs, 4), dtype=torch.int32, device="cuda")
    out["status"] = torch.zeros((H * n_seqs,), dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    nb = binding.workspace_bytes(binding.OP_REPAIR, dt, d, H, batch.cu_seqlens)
    ws = torch.empty((nb,), dtype=torch.uint8, device="cuda")
    rc = L.twinkv_repair(kt.data_ptr(), dt, d, H, n_seqs, cu, kt.stride(0), kt.stride(1),
                         rt.data_ptr(), out["s1"].data_ptr(), bud, tau, w, 2, 3,
                         out["stats"].data_ptr(), out["best_all"].data_ptr(),
                         out["arg_all"].data_ptr(), out["best_ret"].data_ptr(),
                         out["arg_ret"].data_ptr(), ws.data_ptr(), nb, stream)
    assert rc == 0
    nb2 = binding.workspace_bytes(binding.OP_TWIN_COUNTS, dt, d, H, batch.cu_seqlens)
    ws2 = torch.empty((nb2,), dtype=torch.uint8, device="cuda")
    rc = L.twinkv_twin_counts(kt.data_ptr(), dt, d, H, n_seqs, cu, kt.stride(0), kt.stride(1), tau,
                              w, out["counts"].data_ptr(), out["status"].data_ptr(), ws2.data_ptr(),
                              nb2, stream)
    assert rc == 0
    torch.cuda.synchronize()
    return {k: host(v) for k, v in out.items()}


@pytest.mark.parametrize("d,dtype,lens", [(128, "bf16", (5000, 700, 33)), (64, "bf16", (4100, 900, 1)),
                                          (64, "f32", (1500, 260)), (128, "f32", (1300, 70)),
                                          (128, "bf16", (3000, 2048, 64, 0, 1024))])
def test_debug_build_matches(d, dtype, lens):
    sp = synth.Spec(name="dbg", config_id=150 + d + len(lens), n_heads=3, lens=tuple(lens), d=d,
                    dtype=dtype, key_recipe="offset", dup_recipe="uniform", dup_frac=0.2,
                    dup_sigma=0.02, budget_frac=0.4, policy_sinks=2, policy_recent=3, tau=0.9,
                    w=32, n_sink=2, n_recent=3, seed=5)
    batch = synth.make_batch(sp)
    kt, rt = to_device(batch.keys, dtype), mask_to_device(batch.retained)
    dt = 0 if dtype == "bf16" else 1
    a = _run(binding.lib(), kt, rt, batch, dt)
    b = _run(_debug_lib(), kt, rt, batch, dt)
    for k in a:
        assert np.array_equal(a[k], b[k]), k
    assert int(a["stats"][:, 2].sum()) > 0

"""The C ABI from plain C: paper_2608_27128_amd/examples/repair_client.c (built by build() next
to the library) runs the repair pass of Sec. 3.4 with device buffers from the HIP runtime,
without Python or torch in the process.  On the GPU its outputs must equal the ctypes
binding's bit for bit on the same inputs, and the oracle's within the parity protocol.  On the
CPU, argument errors come back through the library's host checks before any device work."""
import os
import struct
import subprocess

import numpy as np
import pytest

import oracle
from gpu_util import check_repair, check_scores, host, mask_to_device, to_device
from paper_2608_27128_amd import binding, build, synth

CLIENT = build.CLIENT


def need_client():
    if not os.path.exists(CLIENT):
        pytest.skip("the C example client is not built (run __graft_entry__.build())")


def write_input(path, batch, tau, w, n_sink, n_recent, d=None):
    H, T = batch.retained.shape
    with open(path, "wb") as f:
        f.write(struct.pack("<6i", H, batch.n_seqs, batch.d if d is None else d, w, n_sink,
                            n_recent))
        f.write(struct.pack("<f", tau))
        f.write(np.asarray(batch.cu_seqlens, "<i8").tobytes())
        f.write(np.asarray(batch.budget, "<i8").tobytes())
        f.write(np.ascontiguousarray(batch.keys.view(np.uint16), "<u2").tobytes())
        f.write(np.ascontiguousarray(batch.retained, np.uint8).tobytes())


def read_output(path, H, n_seqs, T):
    raw = open(path, "rb").read()
    n = H * T
    off = 0

    def take(dt, count):
        nonlocal off
        a = np.frombuffer(raw, dt, count, off)
        off += a.nbytes
        return a

    out = {"s1": take(np.uint8, n).reshape(H, T), "stats": take("<i4", H * n_seqs * 4),
           "best_ret": take("<f4", n).reshape(H, T), "arg_ret": take("<i4", n).reshape(H, T),
           "best_all": take("<f4", n).reshape(H, T), "arg_all": take("<i4", n).reshape(H, T)}
    assert off == len(raw)
    return out


def spec(d):
    return synth.Spec(name="c_client", config_id=91, n_heads=3, lens=(900, 0, 1300, 47), d=d,
                      dtype="bf16", key_recipe="offset", dup_recipe="uniform", dup_frac=0.25,
                      dup_sigma=0.02, budget_frac=0.5, policy_sinks=2, policy_recent=3,
                      tau=0.9, w=32, n_sink=2, n_recent=3, seed=9)


def test_client_rejects_unsupported_head_dimension(tmp_path):
    """d = 96 is refused by twinkv_workspace_bytes on the host: exit status 1 and the
    library's message, nothing enqueued (runs without a GPU)."""
    need_client()
    batch = synth.make_batch(spec(64))
    inp = tmp_path / "in.bin"
    write_input(inp, batch, 0.9, 32, 2, 3, d=96)
    r = subprocess.run([CLIENT, str(inp), str(tmp_path / "out.bin")], capture_output=True,
                       text=True, timeout=60)
    assert r.returncode == 1
    assert "twinkv_workspace_bytes" in r.stderr and "dimension" in r.stderr.lower(), r.stderr
    assert not (tmp_path / "out.bin").exists()


@pytest.mark.gpu
@pytest.mark.parametrize("d", [64, 128])
def test_client_matches_binding_and_oracle(tmp_path, d):
    need_client()
    batch = synth.make_batch(spec(d))
    sp = batch.spec
    inp, outp = tmp_path / "in.bin", tmp_path / "out.bin"
    write_input(inp, batch, sp.tau, sp.w, sp.n_sink, sp.n_recent)
    r = subprocess.run([CLIENT, str(inp), str(outp)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and "repair_client ok" in r.stdout, (r.stdout, r.stderr)
    H, T = batch.retained.shape
    c = read_output(outp, H, batch.n_seqs, T)

    ref = binding.repair(to_device(batch.keys, "bf16"), mask_to_device(batch.retained),
                         batch.budget, sp.tau, sp.w, sp.n_sink, sp.n_recent, batch.cu_seqlens)
    for k in ("s1", "stats", "best_ret", "arg_ret", "best_all", "arg_all"):
        g = host(ref[k]).reshape(c[k].shape)
        assert np.array_equal(g.view(np.uint8), c[k].view(np.uint8)), k

    st = c["stats"].reshape(H, batch.n_seqs, 4)
    for h in range(H):
        for s in range(batch.n_seqs):
            a, e = int(batch.cu_seqlens[s]), int(batch.cu_seqlens[s + 1])
            orc = oracle.repair_problem(batch.keys[h, a:e], "bf16", batch.retained[h, a:e],
                                        batch.budget[s], sp.tau, sp.w, sp.n_sink, sp.n_recent)
            check_scores({k: c[k][h, a:e] for k in ("best_all", "arg_all", "best_ret", "arg_ret")},
                         orc, np.arange(e - a), batch.keys[h, a:e], "bf16",
                         batch.retained[h, a:e], sp.w)
            check_repair(c["s1"][h, a:e], st[h, s], c["best_ret"][h, a:e], orc,
                         batch.retained[h, a:e], sp.tau, sp.n_sink, sp.n_recent)

#!/usr/bin/env python3
"""Throughput of the TwinKV hot path on one MI355X.

One step = one full repair pass (``twinkv_repair``) over a whole synthetic KV cache already
resident in HBM: inverse norms and the [S0 | evicted] partition, the fused similarity
contraction with both masked row max/argmax reductions (all keys and retained keys), then
orphan / donor classification, severity selection and the budget-preserving swap.

Default workload: the long anisotropic cache, 36 layers x 8 KV heads x 32768 tokens x d=128
bf16 (288 problems), tau 0.9, w 32, budget floor(0.3 N) + 4 sinks + 128 recent.

Printed: one JSON line with key-pair similarities per second (N^2 ordered pairs per problem
per step) as ``value``, ms per step (= repair ms per cache), the similarity kernel's roofline
position (its duration measured live with HIP events on the launch stream) and the CPU oracle
timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E
SIM_SOURCE = os.path.join(ROOT, "paper_2608_27128_amd", "csrc", "kernels", "sim_reduce.hip")
COMPACT_SOURCE = os.path.join(ROOT, "paper_2608_27128_amd", "csrc", "kernels", "compact.hip")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


class HipEvents:
    """Raw hipEvent_t handles (created and read through the HIP runtime): the library records
    them on its launch stream around the similarity kernel."""

    def __init__(self):
        import ctypes
        self.ct = ctypes
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def create(self):
        e = self.ct.c_void_p()
        if self.hip.hipEventCreate(self.ct.byref(e)) != 0:
            raise RuntimeError("hipEventCreate failed")
        return e

    def elapsed_ms(self, a, b) -> float:
        ms = self.ct.c_float()
        if self.hip.hipEventElapsedTime(self.ct.byref(ms), a, b) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return float(ms.value)

    def destroy(self, e):
        self.hip.hipEventDestroy(e)


def profiled_traffic(workload: str, name: str = "repair_pass", kernel: str = "sim_reduce",
                     source: str = SIM_SOURCE):
    """HBM bytes per launch of a kernel from the committed rocprofv3 summary
    profiles/<name>_<workload>.md (FETCH_SIZE + WRITE_SIZE, calibrated against a copy of known
    size), or None when no summary exists for this workload or the kernel source has changed
    since it was taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"{name}_{workload}.md")
    if not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        if ":" in line and not line.startswith(("|", "#", "`")):
            k, _, v = line.partition(":")
            fields[k.strip()] = v.strip()
    with open(source, "rb") as f:
        digest = hashlib.sha256(f.read()).hexdigest()[:16]
    if fields.get("workload") != workload or fields.get(f"{kernel}_source_sha256_16") != digest:
        return None
    try:
        return float(fields[f"{kernel}_traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def host_cpu() -> dict:
    """The host the CPU baseline ran on: model name and the CPUs this process may use."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover - not Linux
        usable = os.cpu_count() or 1
    return {"cpu_model": model, "cpus_usable": usable}


def cpu_baseline(batch, target_s: float = 15.0) -> dict:
    """The fp64 oracle on a bounded sample of the same workload: whole problems (all rows,
    both reductions) in (head, sequence) order, then a row prefix of the next one, until
    about target_s seconds of CPU work have been done."""
    import numpy as np
    import oracle
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover - threadpoolctl missing
        cores = os.cpu_count() or 1
    w = batch.spec.w
    H, S = batch.n_heads, batch.n_seqs
    pairs, done, spent = 0.0, [], 0.0
    rate = None
    for q in range(H * S):
        h, s = divmod(q, S)
        a, e = int(batch.cu_seqlens[s]), int(batch.cu_seqlens[s + 1])
        n = e - a
        if n == 0:
            continue
        keys, ret = batch.keys[h, a:e], batch.retained[h, a:e]
        left = target_s - spent
        rows = n if rate is None else int(min(n, max(1, left * rate / n)))
        t = time.perf_counter()
        oracle.nn_scores(keys, batch.dtype, ret, w, rows=np.arange(rows))
        dt = time.perf_counter() - t
        spent += dt
        pairs += rows * n
        rate = pairs / spent
        done.append(f"(h{h},s{s}) rows 0..{rows - 1} of {n}")
        if spent >= 0.9 * target_s:
            break
    return {"value": pairs / spent, "unit": "pairs/s", "cores": int(cores), "kind": "oracle",
            **host_cpu(),
            "sample": f"oracle.nn_scores (both reductions, fp64), d={batch.d}: "
                      f"{'; '.join(done[:3])}{' ...' if len(done) > 3 else ''} "
                      f"({len(done)} problems), {pairs:.3e} ordered pairs in {spent:.1f} s"}


def compact_cpu_baseline(batch, values_of, s1, target_s: float = 10.0) -> dict:
    """oracle.compact_problem on whole problems in (head, sequence) order for about target_s
    seconds; algorithmic bytes as for the GPU kernel."""
    import numpy as np
    import oracle
    H, S = batch.n_heads, batch.n_seqs
    nbytes, spent, done = 0.0, 0.0, 0
    row = batch.keys.shape[2] * batch.keys.itemsize
    for q in range(H * S):
        h, s = divmod(q, S)
        a, e = int(batch.cu_seqlens[s]), int(batch.cu_seqlens[s + 1])
        cap = int(batch.budget[s])
        v = values_of(batch.keys[h, a:e])
        t = time.perf_counter()
        r = oracle.compact_problem(batch.keys[h, a:e], v, s1[h, a:e], cap)
        spent += time.perf_counter() - t
        kept = int(r["stats"][0])
        nbytes += (e - a) + 4.0 * kept * row + 4.0 * cap
        done += 1
        if spent >= target_s:
            break
    return {"value": nbytes / spent / 1e9, "unit": "GB/s", "cores": 1, "kind": "oracle",
            **host_cpu(),
            "sample": f"oracle.compact_problem on {done} whole problems of {H * S} "
                      f"(keys and values, {row}-byte rows), {nbytes / 1e9:.2f} GB in {spent:.1f} s"}


def compact_bench(args, sp, batch, keys, ret, dev) -> int:
    """KV compaction of the keys and values at S1 (Sec. 3.1), S1 produced by one untimed
    repair pass.  Value vectors: the key bits XOR a fixed pattern (any bits are valid rows).
    Algorithmic bytes per step: the mask once, every kept row of keys and values read and
    written once, one int32 position per reserved row."""
    import numpy as np
    import torch
    from paper_2608_27128_amd import binding
    cu = batch.cu_seqlens
    H, T = batch.retained.shape
    rep = binding.repair(keys, ret, batch.budget, sp.tau, sp.w, sp.n_sink, sp.n_recent, cu,
                         want_all=False)
    s1 = rep["s1"]
    ibits = torch.int16 if keys.dtype == torch.bfloat16 else torch.int32
    pattern = 0x5A5A if ibits == torch.int16 else 0x5A5A5A5A
    vals = (keys.view(ibits) ^ pattern).view(keys.dtype)
    cap = np.asarray(batch.budget, dtype=np.int64)
    ws = torch.empty((binding.workspace_bytes(binding.OP_COMPACT, 0, batch.d, H, cu),),
                     dtype=torch.uint8, device=dev)

    def step(outputs=None):
        return binding.compact(keys, s1, cap, values=vals, cu_seqlens=cu, outputs=outputs,
                               workspace=ws)
    out = step()
    for _ in range(args.warmup):
        step(out)
    torch.cuda.synchronize()
    hev = HipEvents()
    g0 = [hev.create() for _ in range(args.steps)]
    g1 = [hev.create() for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for k in range(args.steps):
        binding.profile_sim_events(g0[k], g1[k])
        step(out)
    binding.profile_sim_events(None, None)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    ms_per_step = 1000.0 * wall / args.steps
    g_ms = float(np.mean([hev.elapsed_ms(a, b) for a, b in zip(g0, g1)]))
    for e in g0 + g1:
        hev.destroy(e)
    stats = out["stats"].cpu().numpy()
    assert (stats[:, 2] == 0).all(), "a problem kept more rows than its capacity"
    kept = float(stats[:, 0].sum())
    row = batch.d * (2 if batch.dtype == "bf16" else 4)
    nbytes = float(H * T) + 4.0 * kept * row + 4.0 * H * float(cap.sum())
    log(f"[bench] compact {args.steps} steps: {ms_per_step:.3f} ms/step; gather kernel "
        f"{g_ms:.3f} ms; {kept:.0f} rows kept; {nbytes / 1e9:.3f} GB algorithmic")
    achieved = nbytes / (g_ms * 1e-3) / 1e9
    result = {
        "metric": "KV compaction: algorithmic HBM bytes per second (keys and values at S1)",
        "value": nbytes / (ms_per_step * 1e-3) / 1e9,
        "unit": "GB/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if batch.dtype == "bf16" else "f32", "data": "synthetic",
        "config": {"workload": sp.name, "problems": int(sp.n_heads * sp.n_seqs), "d": int(batch.d),
                   "rows_per_problem": int(cap[0]), "path": "compact", "parallelism": "none"},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": achieved / PEAK_HBM_GBS,
                     "traffic": profiled_traffic(sp.name, "compact", "compact", COMPACT_SOURCE),
                     "kernel": "compact_gather_kernel", "kernel_ms": g_ms,
                     "bytes_per_launch": nbytes},
    }
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a bounded sample ...")
        if batch.dtype == "bf16":
            def values_of(k):
                return k ^ np.uint16(pattern)
        else:
            def values_of(k):
                return (k.view(np.uint32) ^ np.uint32(pattern)).view(np.float32)
        result["cpu_baseline"] = compact_cpu_baseline(batch, values_of, s1.cpu().numpy(),
                                                      min(args.cpu_seconds, 10.0))
    print(json.dumps(result), flush=True)
    return 0


def pipeline_bench(args, sp, batch, keys, dev) -> int:
    """The eviction pipeline end to end on the GPU: a wrapped policy's per-token scores ->
    S0 (twinkv_select_topk, Sec. 3.1 / 3.2) -> the repair pass against the retained columns
    (Sec. 3.4, only b is needed) -> S1 -> the compacted keys and values (Sec. 3.1).  Scores
    are seeded U(0,1) draws on the device, the synthetic policy's distribution.  Value
    vectors as in the compaction bench.  The timed step is the three calls."""
    import numpy as np
    import torch
    from paper_2608_27128_amd import binding
    cu = batch.cu_seqlens
    H, T = batch.retained.shape
    gen = torch.Generator(device=dev)
    gen.manual_seed(0)
    scores = torch.rand((H, T), generator=gen, device=dev, dtype=torch.float32)
    ibits = torch.int16 if keys.dtype == torch.bfloat16 else torch.int32
    pattern = 0x5A5A if ibits == torch.int16 else 0x5A5A5A5A
    vals = (keys.view(ibits) ^ pattern).view(keys.dtype)
    cap = np.asarray(batch.budget, dtype=np.int64)
    dt_code = 0 if batch.dtype == "bf16" else 1
    ws = torch.empty((max(binding.workspace_bytes(binding.OP_REPAIR, dt_code, batch.d, H, cu),
                          binding.workspace_bytes(binding.OP_COMPACT, 0, batch.d, H, cu)),),
                     dtype=torch.uint8, device=dev)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4 * args.steps)]

    def step(outs=None, k=None):
        o = outs or {}
        if k is not None:
            ev[4 * k].record()
        o["sel"] = binding.select_topk(scores, cap, sp.n_sink, sp.n_recent, cu, workspace=ws,
                                       outputs=o.get("sel"))
        if k is not None:
            ev[4 * k + 1].record()
        o["rep"] = binding.repair(keys, o["sel"]["retained"], cap, sp.tau, sp.w, sp.n_sink,
                                  sp.n_recent, cu, want_all=False, outputs=o.get("rep"),
                                  workspace=ws)
        if k is not None:
            ev[4 * k + 2].record()
        o["comp"] = binding.compact(keys, o["rep"]["s1"], cap, values=vals, cu_seqlens=cu,
                                    outputs=o.get("comp"), workspace=ws)
        if k is not None:
            ev[4 * k + 3].record()
        return o
    out = step()
    for _ in range(args.warmup):
        step(out)
    torch.cuda.synchronize()
    hev = HipEvents()
    k0 = [hev.create() for _ in range(args.steps)]
    k1 = [hev.create() for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for k in range(args.steps):
        binding.profile_sim_events(k0[k], k1[k])     # K2 of the repair (compact: its gather)
        step(out, k)
    binding.profile_sim_events(None, None)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    ms_per_step = 1000.0 * wall / args.steps
    stage = np.array([[ev[4 * k + i].elapsed_time(ev[4 * k + i + 1]) for i in range(3)]
                      for k in range(args.steps)])
    k_ms = [hev.elapsed_ms(a, b) for a, b in zip(k0, k1)]
    for e in k0 + k1:
        hev.destroy(e)
    assert (out["sel"]["stats"][:, 0].cpu().numpy() == np.repeat(cap[None, :], H, 0).ravel()).all()
    assert (out["rep"]["stats"][:, 3].cpu().numpy() == 0).all()
    assert (out["comp"]["stats"][:, 2].cpu().numpy() == 0).all()
    sel_ms, rep_ms, comp_ms = (float(x) for x in np.median(stage, axis=0))
    lens = np.diff(cu).astype(np.float64)
    flops = 2.0 * batch.d * sp.n_heads * float(np.sum(lens * cap))     # retained columns only
    # the last profiled span of a step is the compaction's gather; K2 is timed by its stage
    achieved = flops / (rep_ms * 1e-3) / 1e12
    log(f"[bench] pipeline {args.steps} steps: {ms_per_step:.3f} ms/step; select {sel_ms:.3f} ms, "
        f"repair {rep_ms:.3f} ms, compact {comp_ms:.3f} ms (medians of per-stage events)")
    result = {
        "metric": "eviction pipeline (policy scores -> S0 -> repair -> S1 -> compacted K/V): "
                  "cache tokens per second",
        "value": float(H * T) / (ms_per_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if batch.dtype == "bf16" else "f32", "data": "synthetic",
        "config": {"workload": sp.name, "problems": int(sp.n_heads * sp.n_seqs),
                   "d": int(batch.d), "budget": int(cap[0]), "path": "pipeline",
                   "parallelism": "none"},
        "stage_ms": {"select_topk": sel_ms, "repair_retained_columns": rep_ms,
                     "compact": comp_ms},
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS, "traffic": None,
                     "kernel": "repair pass (K1a + K1b + K2 on the retained columns + K3)",
                     "kernel_ms": rep_ms, "flops_per_launch": flops,
                     "gather_ms": float(np.median(k_ms))},
    }
    print(json.dumps(result), flush=True)
    return 0


def sweep_bench(args, sp, keys, dev) -> int:
    """The budget x threshold grid of one policy (Sec. 3.4 repair per cell): the three nested
    retained sets' b in one twinkv_nn_scores_levels call (similarity work N * |S_3| per
    problem), then classification / ranking / swap per (budget, tau) cell from those scores.
    For comparison, the same grid through one retained-only repair pass per budget (work
    N * (|S_1| + |S_2| + |S_3|)) is timed as well."""
    import numpy as np
    import torch
    from paper_2608_27128_amd import binding, synth
    fracs, taus = synth.QWEN_SWEEP_BUDGETS, synth.QWEN_SWEEP_TAUS
    sets = [synth.make_batch(sp, budget_frac=f, threads=min(16, os.cpu_count() or 1)) for f in fracs]
    cu = sets[0].cu_seqlens
    level_np = np.zeros(sets[0].retained.shape, np.uint8)
    for k in range(len(fracs), 0, -1):
        level_np[sets[k - 1].retained != 0] = k
    level = torch.from_numpy(level_np).to(dev)
    rets = [torch.from_numpy(b.retained).to(dev) for b in sets]
    budgets = [b.budget for b in sets]
    H, T = level_np.shape
    lens = np.diff(cu).astype(np.float64)
    s_last = float(np.sum(lens * np.asarray(budgets[-1], dtype=np.float64)))
    pairs = float(H) * s_last                              # N * |S_3| per problem
    flops = 2.0 * keys.shape[2] * pairs
    lv_out = binding.nn_scores_levels(keys, level, len(fracs), sp.w, cu)
    dt_code = binding.TWINKV_BF16 if keys.dtype == torch.bfloat16 else binding.TWINKV_F32
    ws = torch.empty((binding.levels_workspace_bytes(dt_code, keys.shape[2], H, cu, len(fracs),
                                                     False),), dtype=torch.uint8, device=dev)

    def grid():
        out = binding.nn_scores_levels(keys, level, len(fracs), sp.w, cu, workspace=ws,
                                       outputs=lv_out)
        cells = []
        for k in range(len(fracs)):
            for tau in taus:
                cells.append(binding.repair_from_scores(out["best_lvl"][k], rets[k], budgets[k],
                                                        tau, sp.n_sink, sp.n_recent, cu))
        return cells

    def grid_separate():
        cells = []
        for k in range(len(fracs)):
            r = binding.repair(keys, rets[k], budgets[k], taus[0], sp.w, sp.n_sink, sp.n_recent,
                               cu, want_all=False)
            cells.append(r)
            for tau in taus[1:]:
                cells.append(binding.repair_from_scores(r["best_ret"], rets[k], budgets[k], tau,
                                                        sp.n_sink, sp.n_recent, cu))
        return cells

    for _ in range(args.warmup):
        grid()
        grid_separate()
    torch.cuda.synchronize()
    hev = HipEvents()
    e0 = [hev.create() for _ in range(args.steps)]
    e1 = [hev.create() for _ in range(args.steps)]
    t0 = time.perf_counter()
    for k in range(args.steps):
        binding.profile_sim_events(e0[k], e1[k])
        cells = grid()
    binding.profile_sim_events(None, None)
    torch.cuda.synchronize()
    ms = 1000.0 * (time.perf_counter() - t0) / args.steps
    k2_ms = float(np.mean([hev.elapsed_ms(a, b) for a, b in zip(e0, e1)]))
    for e in e0 + e1:
        hev.destroy(e)
    t0 = time.perf_counter()
    for k in range(args.steps):
        cells_sep = grid_separate()
    torch.cuda.synchronize()
    ms_sep = 1000.0 * (time.perf_counter() - t0) / args.steps
    for a, b in zip(cells, cells_sep):     # the same retained sets either way
        assert torch.equal(a["s1"], b["s1"]) and torch.equal(a["stats"], b["stats"])
    log(f"[bench] sweep {args.steps} steps: {ms:.3f} ms per 9-cell grid (similarity sweeps "
        f"{k2_ms:.3f} ms); through one repair pass per budget: {ms_sep:.3f} ms")
    achieved = flops / (k2_ms * 1e-3) / 1e12
    result = {
        "metric": "budget x tau grid (3 x 3 cells) of repair passes: key pairs per second of the "
                  "similarity work it needs (N * |S_3| per problem); ms per grid",
        "value": pairs / (ms * 1e-3), "unit": "pairs/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16" if keys.dtype == torch.bfloat16 else "f32",
        "data": "synthetic",
        "config": {"workload": sp.name, "problems": int(H * (len(cu) - 1)), "d": int(keys.shape[2]),
                   "budgets": [int(b[0]) for b in budgets], "taus": list(taus), "path": "sweep",
                   "parallelism": "none"},
        "grid_ms_one_pass_per_budget": ms_sep,
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS, "traffic": None,
                     "kernel": "sim_reduce_kernel (3 launches, one per level group)",
                     "kernel_ms": k2_ms, "flops_per_launch": flops},
    }
    print(json.dumps(result), flush=True)
    return 0


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=None,
                    help="tiny | llama1b_8k | qwen4b_16k | long_aniso_32k | ragged_64x "
                         "(default long_aniso_32k; qwen4b_16k for --path sweep)")
    ap.add_argument("--path", default="repair",
                    choices=["repair", "repair_s0", "scorer", "compact", "sweep", "pipeline"],
                    help="repair: the full repair pass (both reductions, the headline); "
                         "repair_s0: the repair pass against retained columns only; "
                         "scorer: the standalone scorer (Eq. 2 counts, Eq. 3 eviction); "
                         "compact: KV compaction of the keys and values at S1; "
                         "sweep: the 3 budgets x 3 thresholds grid of the 16k cache; "
                         "pipeline: policy scores -> S0 -> repair -> S1 -> compacted K/V")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="first copy this many MiB device-to-device: a dispatch of known size "
                         "against which memory-traffic counters are scaled")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py: the library runs on exactly one GPU (asked for --gpus {args.gpus}, "
              f"WORLD_SIZE {world}); problems are independent, so more GPUs would each run the "
              f"same single-GPU path on their share of heads.", file=sys.stderr)
        return 2

    import numpy as np
    import torch
    from paper_2608_27128_amd import binding, synth

    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        return 1
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    binding.lib()                                     # fail loudly if the HIP library is missing

    if args.copy_calibration_mib > 0:
        src = torch.ones((args.copy_calibration_mib << 20,), dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        log(f"[bench] calibration copy of {args.copy_calibration_mib} MiB done")

    if args.workload is None:
        args.workload = "qwen4b_16k" if args.path == "sweep" else "long_aniso_32k"
    sp = synth.spec(args.workload)
    if args.path == "sweep":
        keys_sp = synth.make_batch(sp, threads=min(16, os.cpu_count() or 1))
        k = keys_sp.keys
        kt = (torch.from_numpy(k.view(np.int16)).view(torch.bfloat16) if keys_sp.dtype == "bf16"
              else torch.from_numpy(k)).to(dev)
        del keys_sp, k
        return sweep_bench(args, sp, kt, dev)
    t0 = time.perf_counter()
    batch = synth.make_batch(sp, threads=min(16, os.cpu_count() or 1))
    log(f"[bench] generated {sp.name}: keys {batch.keys.shape} {batch.dtype} in "
        f"{time.perf_counter() - t0:.1f} s")

    if batch.dtype == "bf16":
        keys = torch.from_numpy(batch.keys.view(np.int16)).view(torch.bfloat16).to(dev)
    else:
        keys = torch.from_numpy(batch.keys).to(dev)
    ret = torch.from_numpy(batch.retained).to(dev)
    cu = batch.cu_seqlens
    lens = np.diff(cu).astype(np.float64)
    H, T = batch.retained.shape
    dt_code = 0 if batch.dtype == "bf16" else 1
    if args.path == "repair_s0":
        # columns restricted to S0: N * K ordered pairs per problem (K = |S0|)
        pairs = float(sp.n_heads * np.sum(lens * np.asarray(batch.budget, dtype=np.float64)))
    else:
        pairs = float(sp.n_heads * np.sum(lens * lens))  # ordered key pairs per step
    flops = 2.0 * batch.d * pairs                         # dense masked K K^T, per launch

    if args.path == "compact":
        return compact_bench(args, sp, batch, keys, ret, dev)
    if args.path == "pipeline":
        return pipeline_bench(args, sp, batch, keys, dev)

    if args.path in ("repair", "repair_s0"):
        want_all = args.path == "repair"

        def step(outputs=None, ws=None):
            return binding.repair(keys, ret, batch.budget, sp.tau, sp.w, sp.n_sink, sp.n_recent,
                                  cu, want_all=want_all, outputs=outputs, workspace=ws)
        ws = torch.empty((binding.workspace_bytes(binding.OP_REPAIR, dt_code, batch.d, H, cu),),
                         dtype=torch.uint8, device=dev)
    else:
        def step(outputs=None, ws=None):
            return binding.score_evict(keys, batch.budget, sp.tau, sp.w, sp.n_sink, sp.n_recent,
                                       cu, outputs=outputs, workspace=ws)
        ws = torch.empty((binding.workspace_bytes(binding.OP_SCORE_EVICT, dt_code, batch.d, H, cu),),
                         dtype=torch.uint8, device=dev)

    out = step(None, ws)
    for _ in range(args.warmup):
        step(out, ws)
    torch.cuda.synchronize()

    hev = HipEvents()
    k2_start = [hev.create() for _ in range(args.steps)]
    k2_stop = [hev.create() for _ in range(args.steps)]
    # per-step events on the stream the library launches on (torch's current stream)
    st_ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    st_ev[0].record()
    for k in range(args.steps):
        binding.profile_sim_events(k2_start[k], k2_stop[k])
        step(out, ws)
        st_ev[k + 1].record()
    binding.profile_sim_events(None, None)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    ms_per_step = 1000.0 * wall / args.steps
    step_ms = [st_ev[k].elapsed_time(st_ev[k + 1]) for k in range(args.steps)]
    ev_ms = float(np.mean(step_ms))
    k2_each = [hev.elapsed_ms(a, b) for a, b in zip(k2_start, k2_stop)]
    k2_ms = float(np.mean(k2_each))
    for e in k2_start + k2_stop:
        hev.destroy(e)
    stats = out["stats"].cpu().numpy()
    if args.path == "scorer":
        assert (stats[:, 2] == 0).all(), "a problem reported a non-OK status"
        kept = out["retained"].sum(dim=1).cpu().numpy()
        log(f"[bench] {args.steps} steps: {ms_per_step:.3f} ms/step (events {ev_ms:.3f}); "
            f"similarity kernel (count mode) {k2_ms:.3f} ms; kept per head "
            f"{int(kept.min())}..{int(kept.max())}")
    else:
        assert (stats[:, 3] == 0).all(), "a problem reported a non-OK status"
        s1_sum = out["s1"].sum(dim=1).cpu().numpy()
        log(f"[bench] {args.steps} steps: {ms_per_step:.3f} ms/step (events {ev_ms:.3f}); "
            f"similarity kernel {k2_ms:.3f} ms; swaps {int(stats[:, 2].sum())}; "
            f"|S1| per head {int(s1_sum.min())}..{int(s1_sum.max())}")

    achieved = flops / (k2_ms * 1e-3) / 1e12
    result = {
        "metric": "key-pair sims/sec (TFLOP/s of masked K.K^T, % bf16 MFMA peak); repair ms/cache",
        "value": pairs / (ms_per_step * 1e-3),
        "unit": "pairs/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if batch.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {"workload": sp.name, "problems": int(sp.n_heads * sp.n_seqs),
                   "layers_x_kv_heads": int(sp.n_heads), "seq_lens": sorted(set(int(x) for x in lens))[:4],
                   "d": int(batch.d), "tau": sp.tau, "w": sp.w, "n_sink": sp.n_sink,
                   "n_recent": sp.n_recent, "budget": int(batch.budget[0]), "path": args.path,
                   "parallelism": "none"},
        "repair_ms_per_cache": ms_per_step,
        "step_ms_events": {"median": float(np.median(step_ms)), "min": float(np.min(step_ms)),
                           "max": float(np.max(step_ms))},
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS,
                     "traffic": profiled_traffic(sp.name, "repair_pass" if args.path == "repair"
                                                 else f"{args.path}_pass"),
                     "kernel": "sim_reduce_kernel", "kernel_ms": k2_ms,
                     "kernel_ms_median": float(np.median(k2_each)),
                     "kernel_ms_min": float(np.min(k2_each)),
                     "flops_per_launch": flops},
    }
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a bounded sample ...")
        result["cpu_baseline"] = cpu_baseline(batch, args.cpu_seconds)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())

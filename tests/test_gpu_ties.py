"""Exact ties placed at chosen columns: equal similarities must resolve to the smallest
position (reading of Sec. 3.2 / Eq. 4 where the paper leaves argmax ties open), wherever the
kernel meets the tied candidates.  Exact copies of one key tie exactly, and the parity
protocol exempts such rows from the index check (runner-up margin 0), so the rule is checked
here directly.  The placements cover two copies in one 32-column chunk, in different chunks of
one column tile, in different tiles, in the two lane halves of a chunk, a copy in the window
band (redone by the masked pass) against one in the sweep, and copies split between S0 and the
evicted group (the all-keys result merges the two groups)."""
import numpy as np
import pytest

import oracle
from gpu_util import check_scores, host, mask_to_device, to_device
from paper_2608_27128_amd import binding, synth

pytestmark = pytest.mark.gpu

N = 2048
W = 32
# Groups of positions holding exact copies of one key.  Rows 768 and 1152 start a wave's rows
# for every tile shape, so a copy at row + 40 lies in that wave's window band.
GROUPS = [
    (100, 1000, 1010),        # two copies in one chunk (chunk 31)
    (200, 1100, 1060),        # chunks 33 and 34 of one 128-column tile
    (300, 1282, 1285),        # one chunk, columns 2 and 5 (different lane halves)
    (320, 1292, 1296),        # one chunk, columns 12 and 16 (different lane halves)
    (400, 1500, 2000),        # different tiles
    (768, 808, 1900),         # band copy (808) against a sweep copy
    (1152, 1192, 1250, 240),  # sweep copy (240) against a band copy
    (1700, 1720),             # only inside the window of each other: no tie to resolve
]


def planted(d: int, dtype: str, seed: int):
    rng = np.random.default_rng(seed)
    f = rng.standard_normal((1, N, d)).astype(np.float32)
    keys = synth.bf16_bits(f) if dtype == "bf16" else f
    for g in GROUPS:
        for p in g[1:]:
            keys[0, p] = keys[0, g[0]]
    return keys


def expected(group, p, allowed):
    c = [q for q in group if q != p and abs(q - p) > W and allowed[q]]
    return min(c) if c else None


@pytest.mark.parametrize("d,dtype", [(128, "bf16"), (64, "bf16"), (64, "f32"), (128, "f32")])
@pytest.mark.parametrize("with_s0", [False, True])
def test_exact_ties_resolve_to_smallest_position(d, dtype, with_s0):
    keys = planted(d, dtype, seed=d + (dtype == "f32"))
    retained = None
    if with_s0:
        rng = np.random.default_rng(5)
        retained = (rng.random((1, N)) < 0.3).astype(np.uint8)
        # copies on both sides of the S0 / evicted split, either one the smaller position
        for p in (1010, 1060, 1285, 1296, 2000, 1900, 240):
            retained[0, p] = 1
        for p in (1000, 1100, 1282, 1292, 1500, 808, 1192, 1250):
            retained[0, p] = 0
    kt = to_device(keys, dtype)
    out = binding.nn_scores(kt, mask_to_device(retained) if with_s0 else None, W)
    assert np.all(host(out["status"]) == 0)
    ba, aa = host(out["best_all"])[0], host(out["arg_all"])[0]
    br = host(out["best_ret"])[0] if with_s0 else None
    ar = host(out["arg_ret"])[0] if with_s0 else None
    everything = np.ones(N, bool)
    checked = 0
    for g in GROUPS:
        for p in g:
            e = expected(g, p, everything)
            if e is None:
                assert ba[p] < 0.99 and aa[p] not in g, (p, aa[p], ba[p])
            else:
                assert aa[p] == e and abs(ba[p] - 1.0) < 4e-5, (p, aa[p], ba[p], e)
                checked += 1
            if with_s0:
                e = expected(g, p, retained[0].astype(bool))
                if e is not None:
                    assert ar[p] == e and abs(br[p] - 1.0) < 4e-5, (p, ar[p], br[p], e)
                elif br[p] > 0.99:
                    raise AssertionError((p, ar[p], br[p]))
    assert checked >= 15
    # every other row against the oracle under the parity protocol
    rows = np.setdiff1d(np.arange(N), np.concatenate([np.asarray(g) for g in GROUPS]))
    rows = rows[:: 4]
    orc = oracle.nn_scores(keys[0], dtype, retained[0] if with_s0 else None, W, rows=rows)
    gpu = {"best_all": ba, "arg_all": aa}
    if with_s0:
        gpu.update(best_ret=br, arg_ret=ar)
    check_scores(gpu, orc, rows, keys[0], dtype, retained[0] if with_s0 else None, W)


@pytest.mark.parametrize("d,dtype", [(128, "bf16"), (64, "bf16")])
@pytest.mark.parametrize("tail", [1, 17, 31])
def test_twin_at_last_column_of_each_group(d, dtype, tail):
    """A row's only exact twin is the last column of its group (the last retained position
    for b, the last evicted position for the all-keys result), with that group's last
    32-column chunk holding `tail` real columns and padding after them: the reported
    position is the twin's, never a padding slot."""
    n = 1400
    rng = np.random.default_rng(tail + d)
    f = rng.standard_normal((1, n, d)).astype(np.float32)
    keys = synth.bf16_bits(f) if dtype == "bf16" else f
    n_ret = 32 * 9 + tail                               # S0: 9 full chunks + tail columns
    last_ret = n - 60                                   # the largest retained position
    retained = np.zeros((1, n), np.uint8)
    retained[0, [20, last_ret]] = 1                     # row 20 retained, row 10 evicted
    pool = np.setdiff1d(np.arange(100, last_ret), [last_ret])
    retained[0, rng.choice(pool, n_ret - 2, replace=False)] = 1
    assert retained.sum() == n_ret and retained[0, 10] == 0
    last_ev = n - 1                                     # every position past last_ret is evicted
    assert (n - n_ret) % 32 != 0                        # the evicted group ends mid-chunk too
    # row 10 (evicted) is copied to the last retained position; row 20 (retained) to the last
    # evicted position
    keys[0, last_ret] = keys[0, 10]
    keys[0, last_ev] = keys[0, 20]
    kt = to_device(keys, dtype)
    out = binding.nn_scores(kt, mask_to_device(retained), W)
    ar, br = host(out["arg_ret"])[0], host(out["best_ret"])[0]
    aa, ba = host(out["arg_all"])[0], host(out["best_all"])[0]
    assert ar[10] == last_ret and abs(br[10] - 1.0) < 4e-5, (ar[10], br[10], last_ret)
    assert aa[10] == last_ret and abs(ba[10] - 1.0) < 4e-5
    assert aa[20] == last_ev and abs(ba[20] - 1.0) < 4e-5, (aa[20], ba[20], last_ev)
    # and the whole problem against the oracle
    rows = np.arange(n)[::3]
    orc = oracle.nn_scores(keys[0], dtype, retained[0], W, rows=rows)
    check_scores({"best_all": ba, "arg_all": aa, "best_ret": br, "arg_ret": ar}, orc, rows,
                 keys[0], dtype, retained[0], W)

"""Planted mistakes in the oracle must be caught by at least one pin.

Each mutant is a copy of oracle/twinkv_oracle.py with one plausible mistake
(a wrong comparison, a dropped term, a reversed order, a wrong index) written to
a temporary directory and imported as its own module.  The unmodified oracle
passes every pin (test_oracle_pins.py); here every mutant must fail one.
"""
import importlib.util
import os

import pytest

from oracle_pins import ALL_PINS

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                   "oracle", "twinkv_oracle.py")

MUTANTS = {
    "window_inclusive": ("valid = np.abs(rows[:, None] - j[None, :]) > w",
                         "valid = np.abs(rows[:, None] - j[None, :]) >= w"),
    "window_one_sided": ("valid = np.abs(rows[:, None] - j[None, :]) > w",
                         "valid = (rows[:, None] - j[None, :]) > w"),
    "no_normalise": ("out[nz] = K[nz] / norm[nz, None]", "out[nz] = K[nz]"),
    "norm_not_sqrt": ("norm = np.sqrt(np.sum(K * K, axis=1))", "norm = np.sum(K * K, axis=1)"),
    "retained_ignored": ("valid &= member[None, :].astype(bool)", "pass"),
    "tie_largest_j": ("arg = np.argmax(M, axis=1)",
                      "arg = M.shape[1] - 1 - np.argmax(M[:, ::-1], axis=1)"),
    "sentinel_zero": ("best = np.where(any_valid, best, -1.0)",
                      "best = np.where(any_valid, best, 0.0)"),
    "orphan_le": ("orphan = ~s0 & (b < tau)", "orphan = ~s0 & (b <= tau)"),
    "donor_gt": ("donor = s0 & ~prot & (b >= tau)", "donor = s0 & ~prot & (b > tau)"),
    "donor_unprotected": ("donor = s0 & ~prot & (b >= tau)", "donor = s0 & (b >= tau)"),
    "orphan_order_reversed": ("O = O[np.lexsort((O, b[O]))]", "O = O[np.lexsort((O, -b[O]))]"),
    "donor_order_reversed": ("D = D[np.lexsort((D, -b[D]))]", "D = D[np.lexsort((D, b[D]))]"),
    "orphan_tie_reversed": ("O = O[np.lexsort((O, b[O]))]", "O = O[np.lexsort((-O, b[O]))]"),
    "donor_tie_reversed": ("D = D[np.lexsort((D, -b[D]))]", "D = D[np.lexsort((-D, -b[D]))]"),
    "m_is_max": ("m = min(len(O), len(D))", "m = max(len(O), len(D))"),
    "swap_skips_first": ("s1[O[:m]] = True", "s1[O[1:m + 1]] = True"),
    "recent_off_by_one": ("(idx >= n - n_recent)", "(idx > n - n_recent)"),
    "sink_off_by_one": ("(idx < n_sink)", "(idx <= n_sink)"),
    "zero_norm_nan": ("nz = norm > 0", "nz = norm >= 0"),
    # normalising over the wrong axis (one global scale instead of one per key)
    "norm_wrong_axis": ("norm = np.sqrt(np.sum(K * K, axis=1))",
                        "norm = np.sqrt(np.sum(K * K, axis=0)).max() + 0.0 * K[:, 0]"),
    "decode_truncates": ("k = (np.asarray(keys, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)",
                         "k = (np.asarray(keys, dtype=np.uint16).astype(np.uint32) << 15).view(np.float32)"),
    "nonfinite_allowed": ("if not np.all(np.isfinite(k)):", "if False:"),
    "budget_unchecked": ("if int(s0.sum()) != int(budget):", "if False:"),
    # Eq. 2-3 scorer and the prevalence statistic
    "count_ge": ('out["counts"][a:a + step] = np.sum(valid & (S > tau), axis=1)',
                 'out["counts"][a:a + step] = np.sum(valid & (S >= tau), axis=1)'),
    "count_window_ignored": ('out["counts"][a:a + step] = np.sum(valid & (S > tau), axis=1)',
                             'out["counts"][a:a + step] = np.sum(S > tau, axis=1) - 1'),
    "count_tau_scaled": ('out["counts"][a:a + step] = np.sum(valid & (S > tau), axis=1)',
                         'out["counts"][a:a + step] = np.sum(valid & (S > tau * 0.99), axis=1)'),
    "score_sign": ("return -np.asarray(counts, dtype=np.float64) / float(n)",
                   "return np.asarray(counts, dtype=np.float64) / float(n)"),
    "evict_ascending": ("order = np.lexsort((-pos, -score))", "order = np.lexsort((-pos, score))"),
    "evict_tie_earlier": ("order = np.lexsort((-pos, -score))", "order = np.lexsort((pos, -score))"),
    "evict_unprotected": ("score = np.where(protected_mask(n, n_sink, n_recent), np.inf, redundancy_scores(counts, n))",
                          "score = redundancy_scores(counts, n)"),
    "evict_budget_off_by_one": ("keep[order[:min(budget, n)]] = 1", "keep[order[:min(budget + 1, n)]] = 1"),
    "prevalence_ge": ("np.sum(b > float(t))", "np.sum(b >= float(t))"),
    # the margin band of the counts (bounds for a computation with rounded similarities)
    "band_swapped": ('out["counts_lo"][a:a + step] = np.sum(valid & (S > tau + margin), axis=1)',
                     'out["counts_lo"][a:a + step] = np.sum(valid & (S > tau - margin), axis=1)'),
    "band_scaled": ('out["counts_hi"][a:a + step] = np.sum(valid & (S > tau - margin), axis=1)',
                    'out["counts_hi"][a:a + step] = np.sum(valid & (S > tau - 10 * margin), axis=1)'),
    "band_window_ignored": ('out["counts_hi"][a:a + step] = np.sum(valid & (S > tau - margin), axis=1)',
                            'out["counts_hi"][a:a + step] = np.sum(S > tau - margin, axis=1)'),
    "band_not_strict": ('out["counts_lo"][a:a + step] = np.sum(valid & (S > tau + margin), axis=1)',
                        'out["counts_lo"][a:a + step] = np.sum(valid & (S >= tau + margin), axis=1)'),
    # Sec. 3.1 / 3.2 policy selection (reading R22)
    "select_tie_later": ("order = np.lexsort((pos, -s, nan, ~prot))",
                         "order = np.lexsort((-pos, -s, nan, ~prot))"),
    "select_ascending": ("order = np.lexsort((pos, -s, nan, ~prot))",
                         "order = np.lexsort((pos, s, nan, ~prot))"),
    "select_nan_first": ("order = np.lexsort((pos, -s, nan, ~prot))",
                         "order = np.lexsort((pos, -s, ~nan, ~prot))"),
    "select_unprotected": ("order = np.lexsort((pos, -s, nan, ~prot))",
                           "order = np.lexsort((pos, -s, nan))"),
    "select_protected_by_score": ("s = np.where(prot, np.inf, np.where(nan, 0.0, sc))",
                                  "s = np.where(nan, 0.0, sc)"),
    # Sec. 3.1 compaction
    "compact_reversed": ("keep = np.flatnonzero(np.asarray(retained) != 0)",
                         "keep = np.flatnonzero(np.asarray(retained) != 0)[::-1]"),
    "compact_evicted_rows": ("keep = np.flatnonzero(np.asarray(retained) != 0)",
                             "keep = np.flatnonzero(np.asarray(retained) == 0)"),
    "compact_overflow_truncates": ("ok = n_keep <= capacity", "ok = True; keep = keep[:capacity]"),
    "compact_values_from_keys": ("v_out[:n_keep] = np.asarray(values)[keep]", "v_out[:n_keep] = keys[keep]"),
    "compact_pos_one_based": ("pos[:n_keep] = keep", "pos[:n_keep] = keep + 1"),
    "cut_keys_shifted": ('"orphan_cut": (float(b[O[m - 1]]), float(b[O[m]])) if 0 < m < len(O) else None',
                         '"orphan_cut": (float(b[O[m]]), float(b[O[m]])) if 0 < m < len(O) else None'),
    "cut_when_side_whole": ('"donor_cut": (float(b[D[m - 1]]), float(b[D[m]])) if 0 < m < len(D) else None',
                            '"donor_cut": (float(b[D[m - 1]]), float(b[D[min(m, len(D) - 1)]])) if 0 < m <= len(D) else None'),
    "compact_seq_offset_ignored": ("k_out[h, c0[s]:c0[s + 1]] = r[\"keys\"]",
                                   "k_out[h, :cap[s]] = r[\"keys\"]"),
}


def _load_mutant(name, old, new, tmp_path):
    src = open(SRC).read()
    assert src.count(old) >= 1, f"mutation site for {name!r} not found; update the mutant table"
    path = tmp_path / f"mutant_{name}.py"
    path.write_text(src.replace(old, new, 1))
    spec = importlib.util.spec_from_file_location(f"mutant_{name}", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    old, new = MUTANTS[name]
    mod = _load_mutant(name, old, new, tmp_path)
    failed = []
    for pin in ALL_PINS:
        try:
            pin(mod)
        except Exception as e:  # AssertionError or a crash both count as caught
            failed.append((pin.__name__, type(e).__name__))
    assert failed, f"mutant {name!r} passed every pin"

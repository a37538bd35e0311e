"""The oracle's pins catch plausible mistakes.

Each case plants one mistake in the CPU oracle (a dropped term, a wrong
divisor, an off-by-one index, a reversed tie rule, a missing mask, ...) by
replacing one of its functions for the duration of the test, then runs the
pins that should notice it, from tests/test_oracle_pins.py, test_oracle_mass.py
and test_schedule.py.  At least one of them must fail.  The mistakes live only
here, on the CPU; the oracle itself is untouched.
"""
from __future__ import annotations

import math

import numpy as np
import pytest

import oracle
import oracle.sparstar_oracle as OS
from tests import test_oracle_mass as PM
from tests import test_oracle_pins as PP
from tests import test_schedule as PS


def _plant(monkeypatch, name, fn):
    """Replace oracle function `name` both in the package namespace (what the
    pins call) and in the implementation module (what the oracle calls
    internally)."""
    monkeypatch.setattr(OS, name, fn)
    monkeypatch.setattr(oracle, name, fn)


def _some_pin_fails(pins) -> bool:
    for pin in pins:
        try:
            pin()
        except Exception:  # an assertion, or a shape/value error the mistake provokes
            return True
    return False


# ------------------------------------------------------------------ the mistakes
_part = OS.partition


def pool_by_occupancy(x, b):
    """Divides a partial final block by its real rows instead of the nominal b."""
    x = np.asarray(x, dtype=np.float64)
    n = OS.num_blocks(x.shape[0], b)
    counts = np.array([min(b, x.shape[0] - i * b) for i in range(n)], dtype=np.float64)
    return _part(x, b).sum(axis=1) / counts[:, None]


def pool_drops_partial_block(x, b):
    """Pools only the whole blocks; a partial final block pools to zero."""
    out = _part(np.asarray(x, dtype=np.float64), b).sum(axis=1) / b
    if x.shape[0] % b:
        out[-1] = 0.0
    return out


def scores_without_tau(q_bar, k_bar, d, sel):
    s = np.full((q_bar.shape[0], k_bar.shape[0]), np.nan)
    if sel:
        s[:, sel] = q_bar @ k_bar[sel].T
    return s


def scores_shifted_query(q_bar, k_bar, d, sel):
    """Reads the next query block's pooled vector (an index off by one)."""
    return OS.__dict__["_orig_block_scores"](np.roll(q_bar, -1, axis=0), k_bar, d, sel)


def scores_sqrt_missing(q_bar, k_bar, d, sel):
    """tau = 1/D instead of 1/sqrt(D)."""
    s = np.full((q_bar.shape[0], k_bar.shape[0]), np.nan)
    if sel:
        s[:, sel] = (q_bar @ k_bar[sel].T) / d
    return s


def segment_blocks_contained(token_range, lk, b):
    """Forces only blocks lying wholly inside the range (straddling blocks dropped)."""
    begin, end = token_range
    return {j for j in range(OS.num_blocks(lk, b))
            if begin <= OS.block_token_range(j, lk, b)[0] and OS.block_token_range(j, lk, b)[1] <= end
            and begin < end}


def budget_floor(rho, n_sel):
    if not (0.0 <= rho <= 1.0) or math.isnan(rho):
        raise ValueError("density must lie in [0, 1]")
    return min(n_sel, max(1, math.floor(rho * n_sel)))


def budget_without_min_one(rho, n_sel):
    if not (0.0 <= rho <= 1.0) or math.isnan(rho):
        raise ValueError("density must lie in [0, 1]")
    p = rho * n_sel
    r = round(p)
    return min(n_sel, r if abs(p - r) <= 1e-9 * max(1, n_sel) else math.ceil(p))


def budget_plain_ceil(rho, n_sel):
    """The ceiling of the double product, with no snapping to a near integer."""
    if not (0.0 <= rho <= 1.0) or math.isnan(rho):
        raise ValueError("density must lie in [0, 1]")
    return min(n_sel, max(1, math.ceil(rho * n_sel)))


def keep_ranges_swapped(clip, text, ref):
    """Clip 1 keeps only the text and later clips also keep the reference."""
    if clip < 1:
        raise ValueError("clip index starts at 1")
    return [text] if clip == 1 else [text, ref]


def selectable_without_last(keep_set, lk, b):
    ks = set(keep_set)
    return [j for j in range(OS.num_blocks(lk, b) - 1) if j not in ks]


def support_descending(scores_row, keep_set, sel, k):
    return sorted(set(keep_set) | set(OS.topk_idx(scores_row, sel, k)), reverse=True)


def topk_higher_index_wins(scores_row, sel, k):
    return sorted(sel, key=lambda j: (-scores_row[j], -j))[:k]


def topk_smallest(scores_row, sel, k):
    return sorted(sel, key=lambda j: (scores_row[j], j))[:k]


def support_without_keep(scores_row, keep_set, sel, k):
    return sorted(set(OS.topk_idx(scores_row, sel, k)))


def _attention(mutation):
    """sparse_attention with one step of Eq. (7) changed."""
    def f(q, k, v, lists, b, scale=None):
        q, k, v = (np.asarray(a, dtype=np.float64) for a in (q, k, v))
        lq, d = q.shape
        lk = k.shape[0]
        s = (1.0 / math.sqrt(d)) if scale is None else float(scale)
        if mutation == "ignore_scale":
            s = 1.0 / math.sqrt(d)
        out = np.zeros((lq, v.shape[1]))
        lse = np.full(lq, -np.inf)
        for i in range(OS.num_blocks(lq, b)):
            t0, t1 = OS.block_token_range(i, lq, b)
            if mutation == "unmasked_padding":  # every block counted as b keys, zero rows past L_k
                kp = np.vstack([k, np.zeros((b, d))])
                vp = np.vstack([v, np.zeros((b, v.shape[1]))])
                cols = [u for j in lists[i] for u in range(j * b, (j + 1) * b)]
            else:
                kp, vp = k, v
                cols = [u for j in lists[i] for u in range(*OS.block_token_range(j, lk, b))]
            if not cols:
                continue
            z = s * (q[t0:t1] @ kp[cols].T)
            m = z.max(axis=1, keepdims=True)
            p = np.exp(z - m)
            l = p.sum(axis=1, keepdims=True)
            out[t0:t1] = (p @ vp[cols]) / (1.0 if mutation == "unnormalised" else l)
            lse[t0:t1] = (m + (np.log2(l) if mutation == "lse_log2" else np.log(l)))[:, 0]
            if mutation == "lse_without_max":
                lse[t0:t1] = np.log(l)[:, 0]
        return out, lse
    return f


def retained_mass_of_complement(q, k, lists, b, scale=None):
    """Returns the mass the selection drops instead of the mass it keeps."""
    return 1.0 - OS.__dict__["_orig_retained_mass"](q, k, lists, b, scale)


def token_topk_smallest(q, k, n_tokens, scale=None):
    p = OS._dense_probs(q, k, scale)
    srt = np.sort(p, axis=1)
    n = np.asarray(n_tokens, dtype=np.int64)
    return np.array([srt[t, : max(0, min(int(n[t]), p.shape[1]))].sum() for t in range(p.shape[0])])


def scale_densities_first_scales(scale_lq, finest_rho):
    """Assigns the densities to the coarsest scales instead of the finest."""
    n = len(finest_rho)
    return [finest_rho[i] if i < n else None for i in range(len(scale_lq))]


# ------------------------------------------------------------------ the pins each one should trip
SCORE_PINS = [
    lambda: PP.test_block_score_equals_mean_pairwise_compatibility(40, 56, 8, 4),
    lambda: PP.test_block_score_equals_mean_pairwise_compatibility(33, 70, 16, 3),
    PP.test_pool_partial_block_divides_by_nominal_length,
    PP.test_scores_not_computed_for_keep_blocks,
]
KEEP_PINS = [lambda r=r: PP.test_keep_blocks_table(*r) for r in PP.KEEP_TABLE]
BUDGET_PINS = [lambda r=r: PP.test_budget_table(*r) for r in PP.BUDGET_TABLE]
TOPK_PINS = [PP.test_topk_matches_max_sum_subset_bruteforce, PP.test_topk_ties_prefer_lower_index,
             PP.test_select_tiny_planted_blocks_are_recovered]
ATTN_PINS = [
    lambda: PP.test_sparse_attention_matches_sdpa_with_token_mask(100, 150, 16, 8, None),
    lambda: PP.test_sparse_attention_matches_sdpa_with_token_mask(31, 97, 8, 6, 2.0),
    PP.test_zero_queries_give_mean_of_visible_values,
    PP.test_unit_values_give_unit_output_and_single_key_gives_its_value,
    PP.test_full_budget_sparse_equals_dense,
]
MASS_PINS = [PM.test_retained_mass_closed_form_ragged_last_block, PM.test_token_topk_closed_form_with_ties,
             PM.test_token_topk_is_best_subset_by_brute_force, PM.test_retained_mass_brute_force_per_query,
             PM.test_selection_never_beats_the_token_bound]

MUTANTS = [
    ("pool divides by occupancy", "pool", pool_by_occupancy, SCORE_PINS),
    ("pool drops the partial block", "pool", pool_drops_partial_block, SCORE_PINS),
    ("score without tau", "block_scores", scores_without_tau, SCORE_PINS),
    ("score with tau = 1/D", "block_scores", scores_sqrt_missing, SCORE_PINS),
    ("score reads the next query block", "block_scores", scores_shifted_query, SCORE_PINS),
    ("keep only wholly contained blocks", "segment_blocks", segment_blocks_contained, KEEP_PINS),
    ("clip 1 and later clips swapped", "keep_ranges_for_clip", keep_ranges_swapped,
     [PP.test_keep_ranges_for_clip_eq3]),
    ("selectable set misses the last block", "selectable_blocks", selectable_without_last, KEEP_PINS),
    ("budget floor", "budget_k", budget_floor, BUDGET_PINS),
    ("budget without max(1, .)", "budget_k", budget_without_min_one, BUDGET_PINS),
    ("budget ceil without snapping", "budget_k", budget_plain_ceil, BUDGET_PINS),
    ("top-k ties to the higher index", "topk_idx", topk_higher_index_wins, TOPK_PINS),
    ("top-k of the smallest scores", "topk_idx", topk_smallest, TOPK_PINS),
    ("support without the keep set", "retained_support", support_without_keep, TOPK_PINS),
    ("support in descending order", "retained_support", support_descending, TOPK_PINS),
    ("attention ignores the scale argument", "sparse_attention", _attention("ignore_scale"), ATTN_PINS),
    ("attention counts padding keys", "sparse_attention", _attention("unmasked_padding"), ATTN_PINS),
    ("attention without the 1/l normalisation", "sparse_attention", _attention("unnormalised"), ATTN_PINS),
    ("lse in log2", "sparse_attention", _attention("lse_log2"), ATTN_PINS),
    ("lse without the max", "sparse_attention", _attention("lse_without_max"), ATTN_PINS),
    ("retained mass of the complement", "retained_mass", retained_mass_of_complement, MASS_PINS),
    ("token bound of the smallest weights", "token_topk_mass", token_topk_smallest, MASS_PINS),
]


def test_pins_pass_on_the_oracle_as_written():
    for pins in (SCORE_PINS, KEEP_PINS, BUDGET_PINS, TOPK_PINS, ATTN_PINS, MASS_PINS):
        assert not _some_pin_fails(pins)


@pytest.mark.parametrize("name,fn_name,mutant,pins", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_a_pin_catches(monkeypatch, name, fn_name, mutant, pins):
    monkeypatch.setitem(OS.__dict__, "_orig_block_scores", OS.block_scores)
    monkeypatch.setitem(OS.__dict__, "_orig_retained_mass", OS.retained_mass)
    _plant(monkeypatch, fn_name, mutant)
    assert _some_pin_fails(pins), f"no pin notices: {name}"


def test_schedule_pin_catches_coarsest_scale_assignment(monkeypatch):
    _plant(monkeypatch, "scale_densities", scale_densities_first_scales)
    pins = [getattr(PS, n) for n in dir(PS) if n.startswith("test_") and "oracle" in n]
    assert pins, "the schedule pins are named test_*oracle*"
    assert _some_pin_fails(pins)

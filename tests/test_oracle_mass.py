"""Pins of the oracle's retained-attention-mass functions (Section 4, the
analysis comparing the dense softmax mass a selection keeps against the
token-wise top-K upper bound).

Each pin ties the oracle to something it does not compute itself: closed-form
rational masses for logits planted as logarithms of integer weights, brute
force over every subset of keys on tiny inputs, and the invariants that hold
at any size (full selection keeps everything, empty keeps nothing, the block
selection never beats the best equally many single tokens).
"""
import itertools
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle as O


def _planted(weights, d=4):
    """q, k with scale * q . k_u = ln(w_u) exactly in float64 for scale = D^-1/2:
    softmax weights are then w_u / sum(w)."""
    lk = len(weights)
    q = np.zeros((1, d))
    q[0, 0] = 1.0
    k = np.zeros((lk, d))
    k[:, 0] = [math.log(w) * math.sqrt(d) for w in weights]
    return q, k


def test_retained_mass_closed_form_ragged_last_block():
    # L_k = 11 keys in blocks of 4: {0..3}, {4..7}, {8..10} (last block ragged)
    w = [3, 1, 4, 1, 5, 9, 2, 6, 5, 3, 5]
    q, k = _planted(w)
    tot = Fraction(sum(w))
    for blocks in ([], [0], [1], [2], [0, 2], [1, 2], [0, 1, 2]):
        got = O.retained_mass(q, k, [blocks], 4)
        keys = [u for j in blocks for u in range(4 * j, min(4 * j + 4, len(w)))]
        want = Fraction(sum(w[u] for u in keys)) / tot
        assert got[0] == pytest.approx(float(want), abs=1e-12), blocks


def test_token_topk_closed_form_with_ties():
    w = [3, 1, 4, 1, 5, 9, 2, 6, 5, 3, 5]
    q, k = _planted(w)
    tot = sum(w)
    srt = sorted(w, reverse=True)
    for n in range(0, len(w) + 3):
        got = O.token_topk_mass(q, k, np.array([n]))[0]
        assert got == pytest.approx(sum(srt[: min(n, len(w))]) / tot, abs=1e-12), n


def test_token_topk_is_best_subset_by_brute_force():
    rng = np.random.default_rng(3)
    lq, lk, d = 3, 7, 5
    q = rng.standard_normal((lq, d))
    k = rng.standard_normal((lk, d))
    for t in range(lq):
        z = [sum(q[t, c] * k[u, c] for c in range(d)) / math.sqrt(d) for u in range(lk)]
        den = sum(math.exp(x) for x in z)
        for n in range(lk + 1):
            best = max((sum(math.exp(z[u]) for u in sub) / den for sub in itertools.combinations(range(lk), n)),
                       default=0.0)
            got = O.token_topk_mass(q[t:t + 1], k, np.array([n]))[0]
            assert got == pytest.approx(best, abs=1e-12), (t, n)


def test_retained_mass_brute_force_per_query():
    rng = np.random.default_rng(5)
    lq, lk, d, b = 10, 13, 3, 4
    q = rng.standard_normal((lq, d))
    k = rng.standard_normal((lk, d))
    lists = [[0, 3], [1], [], [2, 3]]
    got = O.retained_mass(q, k, lists, b)
    for t in range(lq):
        z = [sum(q[t, c] * k[u, c] for c in range(d)) / math.sqrt(d) for u in range(lk)]
        den = sum(math.exp(x) for x in z)
        keys = [u for j in lists[t // b] for u in range(j * b, min(j * b + b, lk))]
        assert got[t] == pytest.approx(sum(math.exp(z[u]) for u in keys) / den, abs=1e-12), t


def test_full_and_empty_selection():
    rng = np.random.default_rng(11)
    lq, lk, d, b = 20, 37, 8, 8
    q = rng.standard_normal((lq, d)) * 3
    k = rng.standard_normal((lk, d)) * 3
    n_q, n_k = O.num_blocks(lq, b), O.num_blocks(lk, b)
    np.testing.assert_allclose(O.retained_mass(q, k, [list(range(n_k))] * n_q, b), 1.0, atol=1e-12)
    np.testing.assert_array_equal(O.retained_mass(q, k, [[]] * n_q, b), 0.0)
    np.testing.assert_allclose(O.token_topk_mass(q, k, np.full(lq, lk)), 1.0, atol=1e-12)
    np.testing.assert_array_equal(O.token_topk_mass(q, k, np.zeros(lq, dtype=int)), 0.0)


def test_selection_never_beats_the_token_bound():
    """Any block selection keeps at most what the same number of best single
    keys keep; the Eq. (6) selection of the oracle is one such selection."""
    rng = np.random.default_rng(13)
    lq, lk, d, b = 48, 80, 8, 8
    q = rng.standard_normal((lq, d)) * 2
    k = rng.standard_normal((lk, d)) * 2
    lists, _, _, _ = O.select(q, k, b, 0.3, [(0, 5)])
    mass = O.retained_mass(q, k, lists, b)
    n_tok = np.array([sum(min((j + 1) * b, lk) - j * b for j in lists[t // b]) for t in range(lq)])
    bound = O.token_topk_mass(q, k, n_tok)
    assert np.all(mass <= bound + 1e-12)
    assert np.all((mass >= 0) & (bound <= 1 + 1e-12))


def test_scale_argument():
    w = [1, 2, 3, 4]
    q, k = _planted(w)
    # scale 2 * D^-1/2 squares every weight
    got = O.token_topk_mass(q, k, np.array([1]), scale=2 / math.sqrt(4))[0]
    assert got == pytest.approx(16 / 30, abs=1e-12)

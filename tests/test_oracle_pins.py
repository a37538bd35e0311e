"""Pins of the CPU oracle against facts other than itself (no GPU needed).

Each test ties one oracle function to something it does not compute itself:
the bilinearity identity of Section 5.1 evaluated by brute force over token
pairs, hand-derived closed-form tables for Eq. (3)-(5), brute-force subset
enumeration for the top-k of Eq. (6), torch's float64 scaled_dot_product_attention
under the token mask of Eq. (7), and closed forms of special cases.
"""
import itertools
import math

import numpy as np
import pytest
import torch

import oracle as O

pytestmark = pytest.mark.filterwarnings("ignore::DeprecationWarning")


# ---------------------------------------------------------------- pooling + Eq. (2)
def _brute_block_score(q, k, b, i, j):
    """tau * b^-2 * sum over real token pairs (t in B_i, u in B_j) of q_t . k_u:
    the average pairwise pre-softmax compatibility of Section 5.1, with zero
    padding contributing nothing but still counted in the b^2 divisor."""
    lq, d = q.shape
    lk = k.shape[0]
    tot = 0.0
    for t in range(i * b, min((i + 1) * b, lq)):
        for u in range(j * b, min((j + 1) * b, lk)):
            tot += float(sum(q[t, c] * k[u, c] for c in range(d)))
    return tot / (b * b) / math.sqrt(d)


@pytest.mark.parametrize("lq,lk,b,d", [(40, 56, 8, 4), (33, 70, 16, 3), (16, 16, 16, 2)])
def test_block_score_equals_mean_pairwise_compatibility(lq, lk, b, d):
    rng = np.random.default_rng(7)
    q = rng.standard_normal((lq, d))
    k = rng.standard_normal((lk, d))
    sel = list(range(O.num_blocks(lk, b)))
    s = O.block_scores(O.pool(q, b), O.pool(k, b), d, sel)
    for i in range(O.num_blocks(lq, b)):
        for j in sel:
            assert s[i, j] == pytest.approx(_brute_block_score(q, k, b, i, j), rel=1e-12, abs=1e-14)


def test_pool_partial_block_divides_by_nominal_length():
    # Three real rows in a block of nominal length 4: the mean is (1+2+3)/4, not /3.
    x = np.array([[1.0], [2.0], [3.0], [4.0], [1.0], [2.0], [3.0]])
    np.testing.assert_array_equal(O.pool(x, 4), np.array([[2.5], [1.5]]))


def test_pool_and_score_invariant_to_permutation_within_blocks():
    rng = np.random.default_rng(3)
    b, d = 8, 5
    q = rng.standard_normal((24, d))
    k = rng.standard_normal((40, d))
    perm_q = np.concatenate([rng.permutation(8) + 8 * i for i in range(3)])
    perm_k = np.concatenate([rng.permutation(8) + 8 * i for i in range(5)])
    sel = list(range(5))
    s1 = O.block_scores(O.pool(q, b), O.pool(k, b), d, sel)
    s2 = O.block_scores(O.pool(q[perm_q], b), O.pool(k[perm_k], b), d, sel)
    np.testing.assert_allclose(s1, s2, rtol=1e-12, atol=1e-14)


def test_scores_not_computed_for_keep_blocks():
    rng = np.random.default_rng(0)
    qb, kb = rng.standard_normal((3, 4)), rng.standard_normal((6, 4))
    s = O.block_scores(qb, kb, 4, [0, 2, 5])
    assert np.isnan(s[:, [1, 3, 4]]).all() and np.isfinite(s[:, [0, 2, 5]]).all()
    # the selectable columns are tau * q.k with tau = 4^-1/2 = 0.5, computed by hand here
    assert s[1, 2] == pytest.approx(0.5 * float(np.dot(qb[1], kb[2])), rel=1e-14)


# ---------------------------------------------------------------- Eq. (3)-(4): keep sets
# Hand-derived from J = {j : [j*b, min((j+1)*b, Lk)) meets the range}.
KEEP_TABLE = [
    # (ranges, Lk, b, expected J_keep)
    ([(512, 640)], 1152, 64, [8, 9]),                # aligned text segment of the tiny layout
    ([(0, 128)], 1152, 64, [0, 1]),                  # text first ("listed" layout)
    ([(500, 650)], 1152, 64, [7, 8, 9, 10]),         # unaligned: straddles both ends
    ([(512, 576)], 1152, 64, [8]),                   # ends exactly on a block boundary
    ([(575, 577)], 1152, 64, [8, 9]),                # two tokens across a boundary
    ([(300, 300)], 1152, 64, []),                    # empty range
    ([(1150, 1152)], 1152, 64, [17]),                # last block
    ([(1100, 1101)], 1101, 64, [17]),                # last, partial block (Lk = 1101 -> 18 blocks)
    ([(0, 64), (60, 70)], 1152, 64, [0, 1]),         # overlapping ranges: a union
    ([(72_000, 72_512)], 144_512, 128, [562, 563, 564, 565, 566]),  # 720p Eq. (1) text at b = 128
    ([(72_000, 72_512)], 144_512, 64, list(range(1125, 1133))),     # ... and at b = 64
]


@pytest.mark.parametrize("ranges,lk,b,expected", KEEP_TABLE)
def test_keep_blocks_table(ranges, lk, b, expected):
    assert O.keep_blocks(ranges, lk, b) == expected
    sel = O.selectable_blocks(expected, lk, b)
    assert len(sel) == O.num_blocks(lk, b) - len(expected)
    assert not set(sel) & set(expected)


def test_keep_ranges_for_clip_eq3():
    text, ref = (512, 640), (0, 512)
    assert O.keep_ranges_for_clip(1, text, ref) == [text, ref]
    assert O.keep_ranges_for_clip(2, text, ref) == [text]
    assert O.keep_ranges_for_clip(7, text, ref) == [text]
    # tiny layout: clip 1 keeps text + ref blocks 0..9, leaving the 8 current blocks selectable
    assert O.keep_blocks(O.keep_ranges_for_clip(1, text, ref), 1152, 64) == list(range(10))


# ---------------------------------------------------------------- Eq. (5): budget
BUDGET_TABLE = [
    # (rho, n_sel, k) hand-derived from k = min(n, max(1, ceil(rho n)))
    (0.0, 2250, 1), (1e-6, 2250, 1), (0.1, 2250, 225), (0.25, 2250, 563), (0.5, 2250, 1125),
    (1.0, 2250, 2250), (0.09375, 2250, 211), (0.1875, 2250, 422), (0.625, 2250, 1407),
    (0.0, 16, 1), (1e-6, 16, 1), (0.1, 16, 2), (0.25, 16, 4), (0.5, 16, 8), (1.0, 16, 16),
    (0.0, 1, 1), (0.5, 1, 1), (1.0, 1, 1),
    (0.0, 0, 0), (0.5, 0, 0), (1.0, 0, 0),
    (0.25, 1305, 327), (0.7, 10, 7), (0.3, 10, 3),
    # products a hair above an integer in binary (0.14 * 2250 = 315.00000000000006):
    # the exact decimal product is an integer, so that integer is k
    (0.14, 2250, 315), (0.28, 2250, 630), (0.07, 100, 7), (0.55, 100, 55),
]


@pytest.mark.parametrize("rho,n,k", BUDGET_TABLE)
def test_budget_table(rho, n, k):
    assert O.budget_k(rho, n) == k


@pytest.mark.parametrize("rho", [-0.1, 1.5, float("nan")])
def test_budget_rejects_out_of_range(rho):
    with pytest.raises(ValueError):
        O.budget_k(rho, 10)


# ---------------------------------------------------------------- Eq. (6): top-k
def test_topk_matches_max_sum_subset_bruteforce():
    """With distinct scores, the top-k set is the unique k-subset of J_sel with the
    largest total score; enumerate all subsets to find it."""
    rng = np.random.default_rng(11)
    for trial in range(30):
        n_k = int(rng.integers(3, 10))
        keep = sorted(rng.choice(n_k, size=int(rng.integers(0, 3)), replace=False).tolist())
        sel = [j for j in range(n_k) if j not in keep]
        if not sel:
            continue
        row = rng.standard_normal(n_k)
        for kk in range(1, len(sel) + 1):
            best = max(itertools.combinations(sel, kk), key=lambda c: sum(row[j] for j in c))
            assert sorted(O.topk_idx(row, sel, kk)) == sorted(best)
            a = O.retained_support(row, keep, sel, kk)
            assert a == sorted(set(keep) | set(best))


def test_topk_ties_prefer_lower_index():
    row = np.array([1.0, 3.0, 3.0, 2.0, 3.0, np.nan])
    assert O.topk_idx(row, [0, 1, 2, 3, 4], 2) == [1, 2]
    assert O.topk_idx(row, [0, 1, 2, 3, 4], 4) == [1, 2, 4, 3]
    assert O.retained_support(row, [5], [0, 1, 2, 3, 4], 2) == [1, 2, 5]


def test_select_tiny_planted_blocks_are_recovered():
    """On the tiny workload every query block's 3 planted key blocks must be
    among its 4 selected blocks (the planted offset dominates the score)."""
    from synthetic import TINY, bf16_to_f64, generate_head
    from synthetic.workloads import _band_blocks, _plant_candidates, _rng  # recipe replay

    w = TINY
    q, k, _ = generate_head(w, 0, 0)
    # the configuration's forced context: the text segment
    lists, s, kk, keep = O.select(bf16_to_f64(q), bf16_to_f64(k), w.block, w.density, [w.segments()["text"]])
    assert keep == [8, 9] and kk == 4
    # replay the plant stream to recover the planted blocks
    rp = _rng(w, 0, 0, 3)
    cand = _plant_candidates(w)
    for i in range(O.num_blocks(w.lq, w.block)):
        assert _band_blocks(w, i).size == 0
        planted = rp.choice(cand, size=w.aligned, replace=False)
        assert set(planted.tolist()) <= set(lists[i]), (i, planted, lists[i])
        assert len(lists[i]) == len(keep) + kk


# ---------------------------------------------------------------- Eq. (7): attention
def _sdpa(q, k, v, mask, scale):
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a))[None, None]
    out = torch.nn.functional.scaled_dot_product_attention(
        t(q), t(k), t(v), attn_mask=t(mask), scale=scale)
    z = scale * (t(q) @ t(k).transpose(-1, -2))
    lse = torch.logsumexp(z.masked_fill(~t(mask), float("-inf")), dim=-1)
    return out[0, 0].numpy(), lse[0, 0].numpy()


@pytest.mark.parametrize("lq,lk,b,d,scale", [(100, 150, 16, 8, None), (64, 64, 32, 4, 0.7),
                                             (31, 97, 8, 6, 2.0)])
def test_sparse_attention_matches_sdpa_with_token_mask(lq, lk, b, d, scale):
    rng = np.random.default_rng(5)
    q, k, v = (rng.standard_normal((n, d)) for n in (lq, lk, lk))
    n_q, n_k = O.num_blocks(lq, b), O.num_blocks(lk, b)
    lists = [sorted(rng.choice(n_k, size=int(rng.integers(1, n_k + 1)), replace=False).tolist())
             for _ in range(n_q)]
    o, lse = O.sparse_attention(q, k, v, lists, b, scale)
    mask = O.token_mask(lists, lq, lk, b)
    s = (1.0 / math.sqrt(d)) if scale is None else scale
    o_ref, lse_ref = _sdpa(q, k, v, mask, s)
    np.testing.assert_allclose(o, o_ref, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(lse, lse_ref, rtol=1e-10, atol=1e-12)


def test_dense_attention_matches_sdpa():
    rng = np.random.default_rng(6)
    q, k, v = rng.standard_normal((50, 8)), rng.standard_normal((77, 8)), rng.standard_normal((77, 8))
    o, lse = O.dense_attention(q, k, v)
    o_ref, lse_ref = _sdpa(q, k, v, np.ones((50, 77), bool), 1 / math.sqrt(8))
    np.testing.assert_allclose(o, o_ref, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(lse, lse_ref, rtol=1e-10, atol=1e-12)


def test_full_budget_sparse_equals_dense():
    rng = np.random.default_rng(8)
    q, k, v = rng.standard_normal((70, 8)), rng.standard_normal((130, 8)), rng.standard_normal((130, 8))
    lists, _, kk, keep = O.select(q, k, 16, 1.0, [(0, 10)])
    assert all(l == list(range(O.num_blocks(130, 16))) for l in lists)
    o, lse = O.sparse_attention(q, k, v, lists, 16)
    o_d, lse_d = O.dense_attention(q, k, v)
    np.testing.assert_allclose(o, o_d, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(lse, lse_d, rtol=1e-12, atol=1e-13)


def test_zero_queries_give_mean_of_visible_values():
    rng = np.random.default_rng(9)
    lk, b = 90, 16
    k, v = rng.standard_normal((lk, 4)), rng.standard_normal((lk, 4))
    lists = [[0, 5], [3], [1, 2, 4]]
    o, lse = O.sparse_attention(np.zeros((40, 4)), k, v, lists, b)
    for i, blocks in enumerate(lists):
        rows = [u for j in blocks for u in range(j * b, min((j + 1) * b, lk))]
        for t in range(i * b, min((i + 1) * b, 40)):
            np.testing.assert_allclose(o[t], v[rows].mean(axis=0), rtol=1e-12, atol=1e-14)
            assert lse[t] == pytest.approx(math.log(len(rows)), rel=1e-14)


def test_unit_values_give_unit_output_and_single_key_gives_its_value():
    rng = np.random.default_rng(10)
    q, k = rng.standard_normal((20, 4)), rng.standard_normal((33, 4))
    o, _ = O.sparse_attention(q, k, np.ones((33, 4)), [[0, 2], [1]], 16)
    np.testing.assert_allclose(o, 1.0, rtol=0, atol=1e-14)
    # L_k = 33 with b = 16: block 2 holds the single real key 32
    v = rng.standard_normal((33, 4))
    o, lse = O.sparse_attention(q, k, v, [[2], [2]], 16, scale=0.3)
    np.testing.assert_allclose(o, np.broadcast_to(v[32], o.shape), rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(lse, 0.3 * (q @ k[32]), rtol=1e-14)


def test_empty_list_gives_zero_output_and_minus_inf_lse():
    rng = np.random.default_rng(12)
    q, k, v = rng.standard_normal((16, 4)), rng.standard_normal((16, 4)), rng.standard_normal((16, 4))
    o, lse = O.sparse_attention(q, k, v, [[]], 16)
    assert (o == 0).all() and np.isneginf(lse).all()


def test_bf16_rounding_is_round_to_nearest_even():
    """The generator's bf16 rounding agrees with torch's cast."""
    from synthetic import bf16_bits

    rng = np.random.default_rng(13)
    x = np.concatenate([rng.standard_normal(10000).astype(np.float32) * 10,
                        np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, -0.0, 0.0, 65504.0], np.float32)])
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(bf16_bits(x), ref)

"""GPU parity: the HIP path (through the C ABI) against the float64 CPU oracle.

Small cases are compared element by element; they span several tiles and a
ragged tail.  Tolerances (tests/helpers.py): selection exact where the oracle's
boundary gap exceeds 1e-3 (tie-tolerant otherwise), scores |dS| <= 1e-5(1+|S|),
pooled blocks |d| <= 1e-5, O max-abs <= 1e-2 plus relative Frobenius <= 1e-2 per
head, lse max-abs <= 1e-3.
"""
from __future__ import annotations

import math
import sys
import zlib

import numpy as np
import pytest

import oracle as O
from synthetic import TINY, Workload, bf16_bits, bf16_to_f64, generate
from tests.helpers import (keep_for, LSE_ABS, LSE_ABS_SHARP, O_MAX_ABS, O_MAX_ABS_SHARP, bf16_tensor_to_f64, check_gap_rule, check_output,
                           lists_from_device, lists_to_device, to_dev)

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _ws_views(ws, B, H, n_q, n_k, D):
    """The pooled blocks in the selector workspace (layout in sparstar.h): each
    block is 2^e (hi + lo) with hi and lo fp16 and e an int32 scale.  Returns
    them decoded as float64 arrays, q_bar [B,H,n_q,D] and k_bar [B,H,n_k,D]."""
    al = lambda x: (x + 255) // 256 * 256
    rq, rk = B * H * n_q, B * H * n_k
    off_k = al(rq * D * 4)
    off_qe = off_k + al(rk * D * 4)
    off_ke = off_qe + al(rq * 4)
    raw = ws.cpu().numpy()

    def decode(off, rows, off_e, n):
        hl = raw[off: off + rows * D * 4].view(np.float16).reshape(rows, 2, D).astype(np.float64)
        e = raw[off_e: off_e + rows * 4].view(np.int32).astype(np.float64)
        with np.errstate(all="ignore"):  # forced key blocks are never pooled: their rows hold anything
            return ((hl[:, 0] + hl[:, 1]) * np.exp2(e)[:, None]).reshape(B, H, n, D)

    return decode(0, rq, off_qe, n_q), decode(off_k, rk, off_ke, n_k)


def _times_pow2(bits: np.ndarray, e: int) -> np.ndarray:
    """bf16 bit patterns scaled by 2^e exactly (finite, normal values)."""
    from synthetic.workloads import bf16_bits

    return bf16_bits((bf16_to_f64(bits) * 2.0 ** e).astype(np.float32))


def _run_selector(lib, w: Workload, q, k, keep, budget, with_scores=True, fused=False, pooled=False):
    import torch

    B, H, Lq, D = q.shape
    Lk = k.shape[2]
    n_q, n_k = -(-Lq // w.block), -(-Lk // w.block)
    ws = torch.empty(lib.sparstar_score_workspace_bytes(B, H, Lq, Lk, D, w.block), dtype=torch.uint8,
                     device="cuda")
    scores = torch.full((B, H, n_q, n_k), float("nan"), device="cuda") if with_scores else None
    num, idx = lib.sparstar_score_blocks(q, k, w.block, budget, keep, scores=scores, workspace=ws, fused=fused)
    torch.cuda.synchronize()
    qb, kb = _ws_views(ws, B, H, n_q, n_k, D) if pooled else (None, None)
    return num, idx, scores, qb, kb


SELECTOR_CASES = [
    # name, workload, clip
    ("tiny-eq1", TINY, 2),
    ("tiny-listed", TINY.with_(layout="listed"), 2),
    ("tiny-clip1", TINY, 1),
    ("ragged-d128-b64", TINY.with_(name="r1", head_dim=128, lq=500, l_ref=300, l_text=77, heads=3, seed=7), 2),
    ("ragged-d64-b128", TINY.with_(name="r2", block=128, lq=700, l_ref=515, l_text=130, seed=8), 1),
    ("ragged-d128-b128", TINY.with_(name="r3", head_dim=128, block=128, lq=1000, l_ref=1300, l_text=300,
                                    heads=2, seed=9, density=0.4), 2),
    ("many-tiles", TINY.with_(name="r4", head_dim=128, lq=64 * 70 + 5, l_ref=64 * 60 + 9, l_text=200, heads=2,
                              seed=10, aligned=5, density=0.3), 2),
    # rows held in registers at 16 and 24 keys per lane (513-1024 and 1025-1536 key blocks)
    ("rows-800", TINY.with_(name="r8", heads=1, lq=300, l_ref=64 * 800 - 300 - 128 - 5, l_text=128, seed=14,
                            density=0.3), 2),
    ("rows-1300", TINY.with_(name="r9", heads=1, lq=300, l_ref=64 * 1300 - 300 - 128 - 7, l_text=128, seed=15,
                             density=0.3), 2),
    # more than 3584 key blocks: the rows no longer fit in registers and stream from memory
    ("long-rows", TINY.with_(name="r5", heads=1, lq=200, l_ref=64 * 3650 + 17, l_text=128, seed=11,
                             density=0.2), 2),
    # 2304 key blocks, the most the fused score/select kernel keeps in LDS, and one more
    ("fused-limit", TINY.with_(name="r6", heads=2, lq=64 * 17 + 3, l_ref=64 * 2304 - 64 * 17 - 3 - 128,
                               l_text=128, seed=12, density=0.2), 2),
    ("past-fused-limit", TINY.with_(name="r7", heads=1, lq=200, l_ref=64 * 2304 - 200 - 128 + 1, l_text=128,
                                    seed=13, density=0.2), 2),
]
# long rows crowd the scores together; x8 (exact in bf16) spreads them so that
# some rows have a clear top-k boundary
_SPREAD = {"rows-800", "rows-1300", "long-rows", "fused-limit", "past-fused-limit"}


@pytest.mark.parametrize("name,w,clip", SELECTOR_CASES, ids=[c[0] for c in SELECTOR_CASES])
def test_selector_matches_oracle(gpu_lib, name, w, clip):
    _say(f"[selector] {name}: H={w.heads} D={w.head_dim} b={w.block} Lq={w.lq} Lk={w.lk} clip={clip}")
    qb_, kb_, _ = generate(w)
    if name in _SPREAD:
        qb_, kb_ = _times_pow2(qb_, 3), _times_pow2(kb_, 3)
    keep, keep_ref = keep_for(gpu_lib, w, clip)
    q_d, k_d = to_dev(qb_), to_dev(kb_)
    # pool, score and select kernels, with S written out and without
    num, idx, scores, qbar, kbar = _run_selector(gpu_lib, w, q_d, k_d, keep, w.density, pooled=True)
    lists = lists_from_device(num, idx)
    num_n, idx_n, _, _, _ = _run_selector(gpu_lib, w, q_d, k_d, keep, w.density, with_scores=False)
    assert lists_from_device(num_n, idx_n) == lists
    # scores and selection fused (S kept in LDS), up to 2304 key blocks
    n_k = -(-w.lk // w.block)
    lists_f = None
    if n_k <= gpu_lib.FUSED_MAX_BLOCKS:
        num_f, idx_f, _, _, _ = _run_selector(gpu_lib, w, q_d, k_d, keep, w.density, with_scores=False, fused=True)
        lists_f = lists_from_device(num_f, idx_f)
    s_gpu = scores.cpu().numpy()
    stats = {"exact": 0, "tolerant": 0}
    stats_f = {"exact": 0, "tolerant": 0}
    for h in range(w.heads):
        q = bf16_to_f64(qb_[0, h])
        k = bf16_to_f64(kb_[0, h])
        ol, s_ref, kk, keep_set = O.select(q, k, w.block, w.density, keep_ref)
        sel = O.selectable_blocks(keep_set, w.lk, w.block)
        np.testing.assert_allclose(qbar[0, h], O.pool(q, w.block), rtol=0, atol=1e-5)
        np.testing.assert_allclose(kbar[0, h][sel], O.pool(k, w.block)[sel], rtol=0, atol=1e-5)
        err = np.abs(s_gpu[0, h][:, sel] - s_ref[:, sel])
        assert (err <= 1e-5 * (1 + np.abs(s_ref[:, sel]))).all(), f"head {h}: max |dS| {err.max():.3e}"
        for i, row in enumerate(lists[0][h]):
            stats[check_gap_rule(row, s_ref[i], keep_set, sel, kk)] += 1
        if lists_f is not None:
            for i, row in enumerate(lists_f[0][h]):
                stats_f[check_gap_rule(row, s_ref[i], keep_set, sel, kk)] += 1
    _say(f"[selector] {name}: rows {stats}, fused {stats_f if lists_f is not None else 'n/a'}")
    assert stats["exact"] > 0 and (lists_f is None or stats_f["exact"] > 0)


def test_selector_per_head_budgets_and_edge_budgets(gpu_lib):
    w = TINY.with_(name="budgets", heads=5, seed=21)
    _say("[selector] per-head budgets {0, 1e-6, 0.37, 1, 0.5}")
    qb_, kb_, _ = generate(w)
    keep, keep_ref = keep_for(gpu_lib, w)
    budgets = [0.0, 1e-6, 0.37, 1.0, 0.5]
    num, idx, _, _, _ = _run_selector(gpu_lib, w, to_dev(qb_), to_dev(kb_), keep, budgets, with_scores=False)
    lists = lists_from_device(num, idx)
    for h, rho in enumerate(budgets):
        ol, s_ref, kk, keep_set = O.select(bf16_to_f64(qb_[0, h]), bf16_to_f64(kb_[0, h]), w.block, rho, keep_ref)
        sel = O.selectable_blocks(keep_set, w.lk, w.block)
        for i, row in enumerate(lists[0][h]):
            check_gap_rule(row, s_ref[i], keep_set, sel, kk)


def test_selector_eight_keep_ranges(gpu_lib):
    """The most keep ranges the ABI takes (8), scattered, some straddling block
    boundaries and one touching the ragged last block."""
    w = TINY.with_(name="keep8", heads=2, lq=300, l_ref=64 * 40 + 5, l_text=128, seed=23, density=0.3)
    _say(f"[selector] eight keep ranges: Lk={w.lk}")
    qb_, kb_, _ = generate(w)
    lk = w.lk
    keep = [(0, 10), (130, 140), (250, 390), (700, 700), (1000, 1090), (1500, 1540), (2000, 2100),
            (lk - 3, lk)]
    q_d, k_d = to_dev(qb_), to_dev(kb_)
    for fused in (False, True):
        num, idx, _, _, _ = _run_selector(gpu_lib, w, q_d, k_d, keep, w.density, with_scores=False, fused=fused)
        lists = lists_from_device(num, idx)
        for h in range(w.heads):
            _, s_ref, kk, keep_set = O.select(bf16_to_f64(qb_[0, h]), bf16_to_f64(kb_[0, h]), w.block, w.density,
                                              keep)
            sel = O.selectable_blocks(keep_set, w.lk, w.block)
            for i, row in enumerate(lists[0][h]):
                check_gap_rule(row, s_ref[i], keep_set, sel, kk)


def test_selector_256_heads_with_per_head_budgets(gpu_lib):
    """The most heads the ABI takes (256), each with its own budget: the
    per-head budget table indexes by head through the whole range."""
    w = TINY.with_(name="h256", heads=256, head_dim=64, lq=128, l_ref=64 * 6, l_text=64, seed=29, density=0.5)
    _say("[selector] 256 heads, per-head budgets")
    qb_, kb_, _ = generate(w)
    n_k = -(-w.lk // w.block)
    keep, keep_ref = keep_for(gpu_lib, w)
    budgets = [(h % 9) / 8 for h in range(w.heads)]  # 0, 1/8, ..., 1 repeating
    num, idx, _, _, _ = _run_selector(gpu_lib, w, to_dev(qb_), to_dev(kb_), keep, budgets, with_scores=False)
    num = num.cpu().numpy()
    keep_set = O.keep_blocks(keep_ref, w.lk, w.block)
    n_sel = n_k - len(keep_set)
    for h in range(w.heads):
        assert (num[0, h] == len(keep_set) + O.budget_k(budgets[h], n_sel)).all(), h
    for h in (0, 7, 8, 100, 255):
        _, s_ref, kk, ks = O.select(bf16_to_f64(qb_[0, h]), bf16_to_f64(kb_[0, h]), w.block, budgets[h], keep_ref)
        sel = O.selectable_blocks(ks, w.lk, w.block)
        rows = idx[0, h].cpu().numpy()
        for i in range(rows.shape[0]):
            check_gap_rule(rows[i, : num[0, h, i]].tolist(), s_ref[i], ks, sel, kk)


@pytest.mark.parametrize("split", [True, False], ids=["split", "onepass"])
def test_batch_of_two_end_to_end(gpu_lib, split):
    """B = 2 with per-head budgets: selector (separate and fused) and sparse
    forward per (batch, head) against the oracle."""
    import torch

    w = TINY.with_(name="b2", batch=2, heads=3, head_dim=128, lq=64 * 9 + 7, l_ref=64 * 20 + 1, l_text=128,
                   seed=37, density=0.3)
    _say(f"[batch] B={w.batch} H={w.heads} Lq={w.lq} Lk={w.lk} split={split}")
    qb_, kb_, vb_ = generate(w)
    q, k, v = to_dev(qb_), to_dev(kb_), to_dev(vb_)
    keep, keep_ref = keep_for(gpu_lib, w)
    budgets = [0.2, 0.3, 0.45]
    n_q = -(-w.lq // w.block)
    num, idx = gpu_lib.sparstar_score_blocks(q, k, w.block, budgets, keep)
    nf, xf = gpu_lib.sparstar_score_blocks(q, k, w.block, budgets, keep, fused=True)
    o, lse = gpu_lib.sparstar_sparse_attn_fwd(q, k, v, num, idx, w.block, split=split)
    torch.cuda.synchronize()
    lists, lists_f = lists_from_device(num, idx), lists_from_device(nf, xf)
    og, lg = bf16_tensor_to_f64(o), lse.cpu().numpy().astype(np.float64)
    for b in range(w.batch):
        for h in range(w.heads):
            qh, kh, vh = (bf16_to_f64(x[b, h]) for x in (qb_, kb_, vb_))
            _, s_ref, kk, keep_set = O.select(qh, kh, w.block, budgets[h], keep_ref)
            sel = O.selectable_blocks(keep_set, w.lk, w.block)
            for i in range(n_q):
                check_gap_rule(lists[b][h][i], s_ref[i], keep_set, sel, kk)
                check_gap_rule(lists_f[b][h][i], s_ref[i], keep_set, sel, kk)
            o_ref, l_ref = O.sparse_attention(qh, kh, vh, lists[b][h], w.block)
            check_output(og[b, h][None], o_ref[None], lg[b, h][None], l_ref[None], what=f"b {b} h {h}")


def test_selector_everything_forced(gpu_lib):
    """n_sel = 0: every list is exactly J_keep."""
    import torch

    w = TINY.with_(name="allkeep")
    qb_, kb_, _ = generate(w)
    num, idx, _, _, _ = _run_selector(gpu_lib, w, to_dev(qb_), to_dev(kb_), [(0, w.lk)], 0.5, with_scores=False)
    n_k = -(-w.lk // w.block)
    assert (num.cpu() == n_k).all()
    assert (idx.cpu()[..., :n_k] == torch.arange(n_k, dtype=torch.int32)).all()


def test_selector_ties_prefer_lower_index(gpu_lib):
    """Identical key blocks score identically: the lower indices must win."""
    import torch

    w = TINY.with_(name="ties", heads=1)
    qb_, kb_, _ = generate(w)
    kb_ = kb_.copy()
    blk = w.block
    # blocks 0..3 and 12..15 become copies of block 11 (selectable in the Eq. 1 layout)
    for j in list(range(0, 4)) + list(range(12, 16)):
        kb_[0, 0, j * blk:(j + 1) * blk] = kb_[0, 0, 11 * blk:12 * blk]
    keep, keep_ref = keep_for(gpu_lib, w)
    num, idx, scores, _, _ = _run_selector(gpu_lib, w, to_dev(qb_), to_dev(kb_), keep, 3 / 16)
    lists = lists_from_device(num, idx)[0][0]
    s = scores.cpu().numpy()[0, 0]
    keep_set = O.keep_blocks(keep_ref, w.lk, w.block)
    sel = O.selectable_blocks(keep_set, w.lk, w.block)
    for i, row in enumerate(lists):
        # the GPU's own fp32 scores decide; equal scores must resolve to lower indices
        want = sorted(set(keep_set) | set(O.topk_idx(s[i].astype(np.float64), sel, 3)))
        assert row == want, (i, row, want)
    # the fused kernel computes its own scores (another summation order), but
    # the copies score equally among themselves: whichever number of them it
    # takes must be the lowest indices of the group
    num_f, idx_f, _, _, _ = _run_selector(gpu_lib, w, to_dev(qb_), to_dev(kb_), keep, 3 / 16, with_scores=False,
                                          fused=True)
    group = sorted(list(range(0, 4)) + [11] + list(range(12, 16)))
    for i, row in enumerate(lists_from_device(num_f, idx_f)[0][0]):
        taken = [j for j in row if j in group]
        assert taken == group[: len(taken)], (i, row)
        assert len(row) == len(keep_set) + 3


@pytest.mark.parametrize("n_distinct", [1, 40])
def test_selector_heavy_ties_in_long_rows(gpu_lib, n_distinct):
    """Rows of 2,270 key blocks whose selectable blocks are copies of only
    n_distinct blocks: every row's scores take at most n_distinct values, the
    k-th largest sits inside a tied group of dozens of blocks (or of all of
    them), and the sampled bracket of the register search sees repeated keys.
    The lowest indices of the tied group must be taken, on the GPU's own fp32
    scores (separate kernels) and among the copies (fused kernel)."""
    w = TINY.with_(name=f"heavy-ties-{n_distinct}", heads=1, lq=64 * 6, l_ref=64 * 2270 - 64 * 6 - 128,
                   l_text=128, seed=16)
    qb_, kb_, _ = generate(w)
    kb_ = kb_.copy()
    blk, n_k = w.block, -(-w.lk // w.block)
    assert n_k <= gpu_lib.FUSED_MAX_BLOCKS
    src = [37 + 17 * i for i in range(n_distinct)]
    orig = kb_.copy()  # copy from the original blocks: a source block is itself a member of another group
    for j in range(n_k):
        s0 = src[j % n_distinct]
        if (j + 1) * blk <= w.lk:
            kb_[0, 0, j * blk:(j + 1) * blk] = orig[0, 0, s0 * blk:(s0 + 1) * blk]
    keep, keep_ref = keep_for(gpu_lib, w)
    keep_set = O.keep_blocks(keep_ref, w.lk, w.block)
    sel = O.selectable_blocks(keep_set, w.lk, w.block)
    kk = O.budget_k(w.density, len(sel))
    num, idx, scores, _, _ = _run_selector(gpu_lib, w, to_dev(qb_), to_dev(kb_), keep, w.density)
    s = scores.cpu().numpy()[0, 0]
    for i, row in enumerate(lists_from_device(num, idx)[0][0]):
        want = sorted(set(keep_set) | set(O.topk_idx(s[i].astype(np.float64), sel, kk)))
        assert row == want, (i, len(row), len(want))
    num_f, idx_f, _, _, _ = _run_selector(gpu_lib, w, to_dev(qb_), to_dev(kb_), keep, w.density,
                                          with_scores=False, fused=True)
    groups = {}
    for j in sel:
        groups.setdefault(j % n_distinct if (j + 1) * blk <= w.lk else -1 - j, []).append(j)
    for i, row in enumerate(lists_from_device(num_f, idx_f)[0][0]):
        assert len(row) == len(keep_set) + kk
        for g in groups.values():
            taken = [j for j in row if j in g]
            assert taken == g[: len(taken)], (i, taken[:5], g[:5])


def _attn_case(gpu_lib, w: Workload, lists_h, scale=None, v_override=None, q_override=None, split=True,
               k_override=None, stride=None):
    """Run the sparse forward with given lists on all heads; return GPU and oracle outputs.
    stride (default: the longest list) is the kv_stride of the index tensor."""
    import torch

    qb_, kb_, vb_ = generate(w)
    if v_override is not None:
        vb_ = v_override(vb_)
    if q_override is not None:
        qb_ = q_override(qb_)
    if k_override is not None:
        kb_ = k_override(kb_)
    n_q = -(-w.lq // w.block)
    _assert_splits(gpu_lib, w, split)
    num, idx = lists_to_device([lists_h], n_q, stride)
    q, k, v = to_dev(qb_), to_dev(kb_), to_dev(vb_)
    o, lse = gpu_lib.sparstar_sparse_attn_fwd(q, k, v, num, idx, w.block, softmax_scale=scale or 0.0, split=split)
    torch.cuda.synchronize()
    og, lg = bf16_tensor_to_f64(o), lse.cpu().numpy().astype(np.float64)
    refs = [O.sparse_attention(bf16_to_f64(qb_[0, h]), bf16_to_f64(kb_[0, h]), bf16_to_f64(vb_[0, h]),
                               lists_h[h], w.block, scale) for h in range(w.heads)]
    o_ref = np.stack([r[0] for r in refs])[None]
    l_ref = np.stack([r[1] for r in refs])[None]
    return og, lg, o_ref, l_ref, (qb_, kb_, vb_)


# Every case has at least 16 key blocks (the most key ranges the split path
# takes) and a partial last key block, so the split runs for each of the four
# (D, b) instances; _attn_case asserts that it does.  Their lists are short, so
# they take 8 ranges; test_sixteen_key_ranges_match_oracle widens kv_stride to
# reach the 16-range launch on the same inputs.
ATTN_CASES = [
    ("tiny", TINY),
    ("d128-b64-ragged", TINY.with_(name="a1", head_dim=128, lq=500, l_ref=600, l_text=77, heads=3, seed=17)),
    ("d64-b128-ragged", TINY.with_(name="a2", block=128, lq=700, l_ref=1300, l_text=130, seed=18)),
    ("d128-b128-ragged", TINY.with_(name="a3", head_dim=128, block=128, lq=1000, l_ref=1300, l_text=300,
                                    heads=2, seed=19)),
]


def _assert_splits(lib, w: Workload, split: bool):
    """The split path only runs when the library asks for a workspace."""
    if split:
        n = lib.sparstar_attn_workspace_bytes(w.batch, w.heads, w.lq, w.lk, w.head_dim, w.block)
        assert n > 0, f"{w.name}: split requested but the library asks for no workspace"


def _random_lists(w: Workload, rng, heads=None):
    n_q, n_k = -(-w.lq // w.block), -(-w.lk // w.block)
    out = []
    for _ in range(heads or w.heads):
        hl = []
        for i in range(n_q):
            m = int(rng.integers(1, n_k + 1))
            l = sorted(rng.choice(n_k, size=m, replace=False).tolist())
            if i % 3 == 0 and (n_k - 1) not in l:
                l = sorted(l + [n_k - 1])  # the partial last key block
            hl.append(l)
        out.append(hl)
    return out


@pytest.mark.parametrize("name,w", ATTN_CASES, ids=[c[0] for c in ATTN_CASES])
@pytest.mark.parametrize("sharp", [False, True], ids=["tau", "4tau"])
@pytest.mark.parametrize("split", [True, False], ids=["split", "onepass"])
def test_sparse_attention_matches_oracle(gpu_lib, name, w, sharp, split):
    rng = np.random.default_rng(zlib.crc32(name.encode()) % 1000 + int(sharp))
    lists_h = _random_lists(w, rng)
    scale = 4.0 / math.sqrt(w.head_dim) if sharp else None
    _say(f"[attn] {name} sharp={sharp} split={split}: H={w.heads} D={w.head_dim} b={w.block} Lq={w.lq} Lk={w.lk}")
    og, lg, o_ref, l_ref, _ = _attn_case(gpu_lib, w, lists_h, scale, split=split)
    err = check_output(og, o_ref, lg, l_ref, what=name, max_abs=O_MAX_ABS_SHARP if sharp else O_MAX_ABS,
                       lse_abs=LSE_ABS_SHARP if sharp else LSE_ABS)
    _say(f"[attn] {name}: max |dO| = {err:.2e}")


# Lists that can hold this many keys (kv_stride x block size) or more take 16
# key ranges on the split path, shorter ones 8 (include/sparstar.h).
SIXTEEN_RANGES_FROM_KEYS = 24576


@pytest.mark.parametrize("name,w", ATTN_CASES, ids=[c[0] for c in ATTN_CASES])
def test_sixteen_key_ranges_match_oracle(gpu_lib, name, w):
    """The same lists padded to a kv_stride of 24,576 keys take the 16-range
    split launch; they must meet the oracle as the 8-range launch does."""
    rng = np.random.default_rng(zlib.crc32(name.encode()) % 1000 + 11)
    lists_h = _random_lists(w, rng)
    stride = -(-SIXTEEN_RANGES_FROM_KEYS // w.block)
    _say(f"[attn] 16 ranges {name}: kv_stride={stride}")
    og, lg, o_ref, l_ref, _ = _attn_case(gpu_lib, w, lists_h, stride=stride)
    check_output(og, o_ref, lg, l_ref, what=name)
    og8, lg8, _, _, _ = _attn_case(gpu_lib, w, lists_h, stride=stride - 1)
    check_output(og8, o_ref, lg8, l_ref, what=name + " (8 ranges)")


@pytest.mark.parametrize("name,w", ATTN_CASES, ids=[c[0] for c in ATTN_CASES])
def test_softmax_weights_sum_to_one(gpu_lib, name, w):
    """Invariant of Eq. 7: with the GPU's lse and the oracle's float64 logits, the
    weights exp(s q_t . k_u - lse_t) over the visible keys of each query sum to
    one, within exp(LSE_ABS) - 1 (each lse is within LSE_ABS of the exact value)."""
    rng = np.random.default_rng(zlib.crc32(name.encode()) % 1000 + 7)
    lists_h = _random_lists(w, rng)
    _say(f"[attn] softmax sums {name}")
    _, lg, _, _, (qb_, kb_, _) = _attn_case(gpu_lib, w, lists_h)
    tol = math.exp(LSE_ABS) - 1
    for h in range(w.heads):
        q, k = bf16_to_f64(qb_[0, h]), bf16_to_f64(kb_[0, h])
        z = (q @ k.T) / math.sqrt(w.head_dim)
        vis = O.token_mask(lists_h[h], w.lq, w.lk, w.block)
        tot = np.where(vis, np.exp(z - lg[0, h][:, None]), 0.0).sum(axis=1)
        err = np.abs(tot - 1.0)
        assert err.max() <= tol, f"{name} head {h}: max |sum - 1| = {err.max():.3e}"


def test_end_to_end_tiny_against_oracle(gpu_lib):
    """Selector + sparse forward on the tiny workload, each stage against the oracle."""
    import torch

    w = TINY
    _say("[e2e] tiny")
    qb_, kb_, vb_ = generate(w)
    q, k, v = to_dev(qb_), to_dev(kb_), to_dev(vb_)
    keep, keep_ref = keep_for(gpu_lib, w)
    num, idx = gpu_lib.sparstar_score_blocks(q, k, w.block, w.density, keep)
    o, lse = gpu_lib.sparstar_sparse_attn_fwd(q, k, v, num, idx, w.block)
    torch.cuda.synchronize()
    lists = lists_from_device(num, idx)[0]
    for h in range(w.heads):
        qh, kh, vh = (bf16_to_f64(x[0, h]) for x in (qb_, kb_, vb_))
        ol, s_ref, kk, keep_set = O.select(qh, kh, w.block, w.density, keep_ref)
        assert lists[h] == ol  # tiny: every boundary gap is large
        o_ref, l_ref = O.sparse_attention(qh, kh, vh, ol, w.block)
        check_output(bf16_tensor_to_f64(o)[0, h][None], o_ref[None], lse.cpu().numpy()[0, h][None].astype(np.float64),
                     l_ref[None], what=f"head {h}")


@pytest.mark.parametrize("name,w", ATTN_CASES, ids=[c[0] for c in ATTN_CASES])
@pytest.mark.parametrize("split", [True, False], ids=["split", "onepass"])
def test_dense_attention_matches_oracle(gpu_lib, name, w, split):
    import torch

    _say(f"[dense] {name} split={split}")
    _assert_splits(gpu_lib, w, split)
    qb_, kb_, vb_ = generate(w)
    o, lse = gpu_lib.sparstar_dense_attn_fwd(to_dev(qb_), to_dev(kb_), to_dev(vb_), w.block, split=split)
    torch.cuda.synchronize()
    refs = [O.dense_attention(bf16_to_f64(qb_[0, h]), bf16_to_f64(kb_[0, h]), bf16_to_f64(vb_[0, h]))
            for h in range(w.heads)]
    check_output(bf16_tensor_to_f64(o), np.stack([r[0] for r in refs])[None], lse.cpu().numpy().astype(np.float64),
                 np.stack([r[1] for r in refs])[None], what=name)


@pytest.mark.parametrize("split,long", [(True, False), (True, True), (False, False)],
                         ids=["split", "split-16-ranges", "onepass"])
def test_full_lists_equal_dense(gpu_lib, split, long):
    """rho = 1 (every block listed) equals the dense forward, bit for bit; the
    long case has 24,576 keys and more, so both calls take 16 key ranges."""
    import torch

    w = ATTN_CASES[1][1]
    if long:
        w = w.with_(name="a1-long", heads=1, lq=300, l_ref=SIXTEEN_RANGES_FROM_KEYS + 40 - w.l_text - 300)
        assert w.lk == SIXTEEN_RANGES_FROM_KEYS + 40
    _say(f"[dense==sparse(all)] split={split} Lk={w.lk}")
    _assert_splits(gpu_lib, w, split)
    qb_, kb_, vb_ = generate(w)
    q, k, v = to_dev(qb_), to_dev(kb_), to_dev(vb_)
    n_q, n_k = -(-w.lq // w.block), -(-w.lk // w.block)
    num, idx = lists_to_device([[[list(range(n_k))] * n_q for _ in range(w.heads)]], n_q)
    o1, l1 = gpu_lib.sparstar_sparse_attn_fwd(q, k, v, num, idx, w.block, split=split)
    o2, l2 = gpu_lib.sparstar_dense_attn_fwd(q, k, v, w.block, split=split)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_unit_values_give_unit_output(gpu_lib):
    import torch

    w = ATTN_CASES[1][1]
    _say("[V=1]")
    lists_h = _random_lists(w, np.random.default_rng(3))
    og, lg, o_ref, l_ref, _ = _attn_case(gpu_lib, w, lists_h, v_override=lambda v: np.full_like(v, 0x3F80))
    # the row sum is over the same bf16 P that multiplies V, so the weights sum to one
    assert (og == 1.0).all()


def test_zero_queries_average_selected_values(gpu_lib):
    w = ATTN_CASES[1][1]
    _say("[Q=0]")
    lists_h = _random_lists(w, np.random.default_rng(4))
    og, lg, o_ref, l_ref, _ = _attn_case(gpu_lib, w, lists_h, q_override=lambda q: np.zeros_like(q))
    check_output(og, o_ref, lg, l_ref, what="Q=0")
    n_k = -(-w.lk // w.block)
    for h in range(w.heads):
        for i, l in enumerate(lists_h[h][:3]):
            nkeys = sum(min((j + 1) * w.block, w.lk) - j * w.block for j in l)
            assert lg[0, h, i * w.block] == pytest.approx(math.log(nkeys), abs=1e-5)
    assert n_k > 1


@pytest.mark.parametrize("split", [True, False], ids=["split", "onepass"])
def test_empty_and_invalid_list_entries(gpu_lib, split):
    """Empty rows give O = 0, lse = -inf; out-of-range entries of an ascending list
    are skipped; counts clamp to the stride."""
    import torch

    w = ATTN_CASES[0][1]
    _say(f"[empty/invalid lists] split={split}")
    qb_, kb_, vb_ = generate(w)
    q, k, v = to_dev(qb_), to_dev(kb_), to_dev(vb_)
    n_q, n_k = -(-w.lq // w.block), -(-w.lk // w.block)
    stride = 4
    num = torch.zeros((1, w.heads, n_q), dtype=torch.int32)
    idx = torch.zeros((1, w.heads, n_q, stride), dtype=torch.int32)
    lists_ref = [[[] for _ in range(n_q)] for _ in range(w.heads)]
    for h in range(w.heads):
        for i in range(n_q):
            if i % 3 == 0:
                continue  # empty
            if i % 3 == 1:
                num[0, h, i] = 4
                idx[0, h, i] = torch.tensor([-3, 1, 4, n_k + 5])
                lists_ref[h][i] = [1, 4]
            else:
                num[0, h, i] = 99  # clamped to the stride (4)
                idx[0, h, i] = torch.tensor([0, 2, 7, n_k - 1])
                lists_ref[h][i] = [0, 2, 7, n_k - 1]
    o, lse = gpu_lib.sparstar_sparse_attn_fwd(q, k, v, num.cuda(), idx.cuda(), w.block, split=split)
    torch.cuda.synchronize()
    refs = [O.sparse_attention(bf16_to_f64(qb_[0, h]), bf16_to_f64(kb_[0, h]), bf16_to_f64(vb_[0, h]),
                               lists_ref[h], w.block) for h in range(w.heads)]
    og = bf16_tensor_to_f64(o)
    lg = lse.cpu().numpy().astype(np.float64)
    check_output(og, np.stack([r[0] for r in refs])[None], lg, np.stack([r[1] for r in refs])[None], what="lists")
    assert (og[0, :, : w.block] == 0).all() and np.isneginf(lg[0, :, : w.block]).all()


def test_split_agrees_with_single_pass(gpu_lib):
    """The key-range split and the single pass agree to fp16/fp32 rounding."""
    import torch

    w = ATTN_CASES[3][1]
    _say("[split vs one pass]")
    qb_, kb_, vb_ = generate(w)
    q, k, v = to_dev(qb_), to_dev(kb_), to_dev(vb_)
    num, idx = gpu_lib.sparstar_score_blocks(q, k, w.block, 0.3, keep_for(gpu_lib, w)[0])
    o1, l1 = gpu_lib.sparstar_sparse_attn_fwd(q, k, v, num, idx, w.block, split=True)
    o2, l2 = gpu_lib.sparstar_sparse_attn_fwd(q, k, v, num, idx, w.block, split=False)
    torch.cuda.synchronize()
    # P is rounded relative to each range's own running max, so the two paths
    # round differently; each is within the bf16-P bounds of the exact result
    assert (o1.float() - o2.float()).abs().max().item() <= O_MAX_ABS
    assert (l1 - l2).abs().max().item() <= LSE_ABS


def test_deterministic(gpu_lib):
    import torch

    w = ATTN_CASES[1][1]
    _say("[determinism]")
    qb_, kb_, vb_ = generate(w)
    q, k, v = to_dev(qb_), to_dev(kb_), to_dev(vb_)
    keep, keep_ref = keep_for(gpu_lib, w)
    r1 = gpu_lib.sparstar_score_blocks(q, k, w.block, w.density, keep)
    r2 = gpu_lib.sparstar_score_blocks(q, k, w.block, w.density, keep)
    o1 = gpu_lib.sparstar_sparse_attn_fwd(q, k, v, *r1, w.block)
    o2 = gpu_lib.sparstar_sparse_attn_fwd(q, k, v, *r2, w.block)
    torch.cuda.synchronize()
    assert torch.equal(r1[0], r2[0])
    n = r1[0].cpu()
    i1, i2 = r1[1].cpu(), r2[1].cpu()
    for h in range(w.heads):
        for i in range(n.shape[2]):
            c = int(n[0, h, i])
            assert torch.equal(i1[0, h, i, :c], i2[0, h, i, :c])
    assert torch.equal(o1[0], o2[0]) and torch.equal(o1[1], o2[1])
    # the fused selector too
    f1 = gpu_lib.sparstar_score_blocks(q, k, w.block, w.density, keep, fused=True)
    f2 = gpu_lib.sparstar_score_blocks(q, k, w.block, w.density, keep, fused=True)
    torch.cuda.synchronize()
    assert torch.equal(f1[0], f2[0])
    nf = f1[0].cpu()
    j1, j2 = f1[1].cpu(), f2[1].cpu()
    for h in range(w.heads):
        for i in range(nf.shape[2]):
            c = int(nf[0, h, i])
            assert torch.equal(j1[0, h, i, :c], j2[0, h, i, :c])


def test_empty_query_sequence_is_noop(gpu_lib):
    import torch

    w = TINY
    qb_, kb_, vb_ = generate(w)
    q = torch.empty((1, w.heads, 0, w.head_dim), dtype=torch.bfloat16, device="cuda")
    k, v = to_dev(kb_), to_dev(vb_)
    num, idx = gpu_lib.sparstar_score_blocks(q, k, w.block, 0.25, keep_for(gpu_lib, w)[0])
    o, lse = gpu_lib.sparstar_sparse_attn_fwd(q, k, v, num, idx, w.block)
    torch.cuda.synchronize()
    assert o.numel() == 0 and num.numel() == 0


@pytest.mark.parametrize("e", [20, -20, 60, -60])
@pytest.mark.parametrize("split", [True, False], ids=["split", "onepass"])
def test_value_magnitudes_far_outside_fp16(gpu_lib, e, split):
    """V scaled by 2^e (exact in bf16): Eq. 7 is linear in V, so O must scale by
    exactly 2^e and lse not at all, on the split path (fp16 partials with a
    per-row power-of-two scale) as on the single pass, and match the oracle.
    |V| reaches about 5 * 2^60 here, far beyond fp16's 65504, and 2^-60 is far
    below its smallest normal."""
    w = ATTN_CASES[1][1]
    _say(f"[V x 2^{e}] split={split}")
    lists_h = _random_lists(w, np.random.default_rng(11))
    og0, lg0, _, _, _ = _attn_case(gpu_lib, w, lists_h, split=split)
    og, lg, o_ref, l_ref, _ = _attn_case(gpu_lib, w, lists_h, split=split, v_override=lambda v: _times_pow2(v, e))
    assert np.array_equal(og, og0 * 2.0 ** e), "O does not scale exactly with V"
    assert np.array_equal(lg, lg0), "lse depends on the scale of V"
    check_output(og * 2.0 ** -e, o_ref * 2.0 ** -e, lg, l_ref, what=f"V x 2^{e}")


def _group_offsets(n_groups: int) -> np.ndarray:
    """Logit offset (about one unit = one binade at D = 128) of each 32-key
    group: in every run of four groups a rise of 20, a fall to +5, a fall to
    -10, on a base that climbs 6 per run, and from group 50 on everything 150
    higher (a jump past 2^128)."""
    g = np.arange(n_groups)
    c = 6.0 * (g // 4) + np.array([0.0, 20.0, 5.0, -10.0])[g % 4]
    return c + np.where(g >= 50, 150.0, 0.0)


@pytest.mark.parametrize("block", [64, 128])
@pytest.mark.parametrize("split", [True, False], ids=["split", "onepass"])
def test_running_max_jumps(gpu_lib, block, split):
    """Logits that rise along every list by a few, by tens and, once, by 150
    binades (Eq. 7's softmax over them).  The kernel forms P against its
    running max and moves that max only when a 32-key sub-tile's P could pass
    2^8: small rises stay on the fast path with p up to 2^8, larger ones take
    the exact path (a power-of-two rescale of O and both row sums, and at
    b = 128 of the bf16 P of the step's first sub-tile when its second one
    rises), and the 150-binade jump drops the old terms.  O and lse must match
    the oracle as on ordinary inputs."""
    w = TINY.with_(name="jumps", head_dim=128, block=block, lq=300, l_ref=1700, l_text=200, heads=2, seed=23)
    rng = np.random.default_rng(29 + block)

    def q_over(qb):
        q = 0.25 + 0.02 * rng.standard_normal(qb.shape).astype(np.float32)
        return bf16_bits(q)

    def k_over(kb):
        n_groups = -(-w.lk // 32)
        c = np.repeat(_group_offsets(n_groups), 32)[: w.lk].astype(np.float32)
        k = rng.standard_normal(kb.shape).astype(np.float32) + 0.25 * c[None, None, :, None]
        return bf16_bits(k)

    lists_h = _random_lists(w, np.random.default_rng(31 + block))
    lists_h[0][0] = list(range(-(-w.lk // w.block)))  # one query block sees every key block
    _say(f"[jumps] b={block} split={split}")
    og, lg, o_ref, l_ref, _ = _attn_case(gpu_lib, w, lists_h, split=split, q_override=q_over, k_override=k_over)
    assert np.isfinite(og).all() and np.isfinite(lg).all()
    # the logits reach about 300 binades: lse is large, and its fp32 value is
    # compared at the same absolute tolerance as everywhere else
    assert l_ref.max() > 150.0
    check_output(og, o_ref, lg, l_ref, what=f"jumps b={block}")


_CANARY = 0x5A  # byte pattern of untouched guard memory


def _guarded(shape, dtype, guard=4096):
    """A contiguous tensor of `shape` inside a canary-filled byte buffer with
    `guard` bytes before and after it; returns (buffer, view, bytes of the view)."""
    import torch

    n = int(np.prod(shape)) * torch.empty((), dtype=dtype).element_size()
    buf = torch.full((guard + n + guard,), _CANARY, dtype=torch.uint8, device="cuda")
    return buf, buf[guard: guard + n].view(dtype).view(*shape), n


def _guards_intact(buf, n, guard=4096):
    b = buf.cpu().numpy()
    return bool((b[:guard] == _CANARY).all() and (b[guard + n:] == _CANARY).all())


@pytest.mark.parametrize("fused", [False, True], ids=["separate", "fused"])
def test_selector_writes_only_its_list_entries(gpu_lib, fused):
    """kv_indices entries past each row's count are left untouched (the header's
    promise), with per-head budgets so that the counts differ between heads and a
    stride wider than needed; nothing outside the two outputs is written."""
    import torch

    w = ATTN_CASES[1][1]
    _say(f"[guard] selector fused={fused}")
    qb_, kb_, _ = generate(w)
    keep, keep_ref = keep_for(gpu_lib, w)
    budgets = [0.1, 0.3, 0.6]
    n_q = -(-w.lq // w.block)
    stride = gpu_lib.sparstar_kv_stride(w.heads, w.lk, w.block, budgets, keep) + 5
    nbuf, num, nn = _guarded((1, w.heads, n_q), torch.int32)
    ibuf, idx, ni = _guarded((1, w.heads, n_q, stride), torch.int32)
    gpu_lib.sparstar_score_blocks(to_dev(qb_), to_dev(kb_), w.block, budgets, keep, kv_stride=stride,
                                  out=(num, idx), fused=fused)
    torch.cuda.synchronize()
    assert _guards_intact(nbuf, nn) and _guards_intact(ibuf, ni), "a write outside the outputs"
    canary = np.frombuffer(bytes([_CANARY] * 4), dtype=np.int32)[0]
    n, ix = num.cpu().numpy(), idx.cpu().numpy()
    keep_set = O.keep_blocks(keep_ref, w.lk, w.block)
    n_sel = -(-w.lk // w.block) - len(keep_set)
    for h, rho in enumerate(budgets):
        c = len(keep_set) + O.budget_k(rho, n_sel)
        assert (n[0, h] == c).all()
        assert (ix[0, h, :, c:] == canary).all(), f"head {h}: an entry past the count was written"
        assert (ix[0, h, :, :c] != canary).all()


@pytest.mark.parametrize("dense", [False, True], ids=["sparse", "dense"])
@pytest.mark.parametrize("split", [True, False], ids=["split", "onepass"])
def test_attention_writes_only_its_outputs(gpu_lib, dense, split):
    """O and lse sit inside canary-filled guard bands; the last query block is
    partial (Lq = 500 at b = 64), so rows past Lq would land in the band after
    the last head.  Nothing outside O and lse changes, and the result matches
    the oracle."""
    import torch

    w = ATTN_CASES[1][1]
    _say(f"[guard] attention dense={dense} split={split}")
    _assert_splits(gpu_lib, w, split)
    qb_, kb_, vb_ = generate(w)
    q, k, v = to_dev(qb_), to_dev(kb_), to_dev(vb_)
    n_q = -(-w.lq // w.block)
    assert w.lq % w.block != 0
    lists_h = _random_lists(w, np.random.default_rng(5))
    obuf, o, no = _guarded((1, w.heads, w.lq, w.head_dim), torch.bfloat16)
    lbuf, lse, nl = _guarded((1, w.heads, w.lq), torch.float32)
    if dense:
        gpu_lib.sparstar_dense_attn_fwd(q, k, v, w.block, out=o, lse=lse, split=split)
        lists_h = [[list(range(-(-w.lk // w.block)))] * n_q for _ in range(w.heads)]
    else:
        num, idx = lists_to_device([lists_h], n_q)
        gpu_lib.sparstar_sparse_attn_fwd(q, k, v, num, idx, w.block, out=o, lse=lse, split=split)
    torch.cuda.synchronize()
    assert _guards_intact(obuf, no), "O: a write outside the output"
    assert _guards_intact(lbuf, nl), "lse: a write outside the output"
    refs = [O.sparse_attention(bf16_to_f64(qb_[0, h]), bf16_to_f64(kb_[0, h]), bf16_to_f64(vb_[0, h]),
                               lists_h[h], w.block) for h in range(w.heads)]
    check_output(bf16_tensor_to_f64(o), np.stack([r[0] for r in refs])[None], lse.cpu().numpy().astype(np.float64),
                 np.stack([r[1] for r in refs])[None], what="guarded")

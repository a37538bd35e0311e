"""GPU parity at the full workload sizes, on sampled outputs the oracle can
compute one by one.

All 24 heads run through the C ABI in the launch configuration the benchmark
times (key-range split with a workspace); the float64 oracle then recomputes
the selector of sampled heads completely (every row checked under the gap
rule) and the forward of sampled query blocks (first, last and interior ones).
At the 720p headline shape every head's forward is checked on four query
blocks, and six heads' selectors on every row.
"""
from __future__ import annotations

import sys

import numpy as np
import pytest

import oracle as O
from synthetic import MID, P720, SWEEP, bf16_to_f64, generate, head_densities, keep_ranges
from tests.helpers import check_gap_rule, check_output, to_dev

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _run_full(lib, w, budget, fused=None):
    """fused: a list that receives the fused selector's (num, idx) as well."""
    import torch

    _say(f"[full] {w.name}: generating H={w.heads} Lq={w.lq} Lk={w.lk}")
    qb, kb, vb = generate(w, workers=1)
    q, k, v = to_dev(qb), to_dev(kb), to_dev(vb)
    keep = keep_ranges(w)
    _say(f"[full] {w.name}: selector + sparse forward on the GPU")
    num, idx = lib.sparstar_score_blocks(q, k, w.block, budget, keep)
    o, lse = lib.sparstar_sparse_attn_fwd(q, k, v, num, idx, w.block)
    if fused is not None:
        _say(f"[full] {w.name}: fused score/select on the GPU")
        nf, xf = lib.sparstar_score_blocks(q, k, w.block, budget, keep, fused=True)
        fused.extend([nf.cpu().numpy(), xf.cpu().numpy()])
    torch.cuda.synchronize()
    return (qb, kb, vb), keep, num.cpu().numpy(), idx.cpu().numpy(), o.float().cpu().numpy(), lse.cpu().numpy()


def _check_heads(w, data, keep, num, idx, o, lse, heads, qblocks, budgets, selector=True):
    """selector=False checks only the forward (on the GPU's own lists)."""
    qb, kb, vb = data
    n_q = -(-w.lq // w.block)
    for h in heads:
        qh, kh, vh = bf16_to_f64(qb[0, h]), bf16_to_f64(kb[0, h]), bf16_to_f64(vb[0, h])
        gpu_lists = [idx[0, h, i, : num[0, h, i]].tolist() for i in range(n_q)]
        if selector:
            rho = float(budgets[h])
            _say(f"[full] {w.name}: oracle selector head {h} (rho={rho:.4f})")
            lists_ref, s_ref, kk, keep_set = O.select(qh, kh, w.block, rho, keep)
            sel = O.selectable_blocks(keep_set, w.lk, w.block)
            stats = {"exact": 0, "tolerant": 0}
            for i in range(n_q):
                stats[check_gap_rule(gpu_lists[i], s_ref[i], keep_set, sel, kk)] += 1
            _say(f"[full] {w.name}: head {h} rows {stats}")
        for i in qblocks:
            rows = slice(i * w.block, min((i + 1) * w.block, w.lq))
            o_ref, l_ref = O.sparse_attention(qh[rows], kh, vh, [gpu_lists[i]], w.block)
            check_output(o[0, h, rows][None].astype(np.float64), o_ref[None], lse[0, h, rows][None].astype(np.float64),
                         l_ref[None], what=f"{w.name} head {h} block {i}")


def test_mid_scale_parity(gpu_lib):
    w = MID
    data, keep, num, idx, o, lse = _run_full(gpu_lib, w, w.density)
    n_q = -(-w.lq // w.block)
    _check_heads(w, data, keep, num, idx, o, lse, heads=[0, 13, 23], qblocks=[0, 1, 90, n_q - 1],
                 budgets=np.full(w.heads, w.density))


def test_720p_final_scale_parity(gpu_lib):
    w = P720
    fused = []
    data, keep, num, idx, o, lse = _run_full(gpu_lib, w, w.density, fused=fused)
    n_q = -(-w.lq // w.block)
    assert (num == 8 + 563).all()
    # every head: four query blocks of the forward, stratified so that the first and last blocks are always
    # checked and the other two move across the sequence; every fifth head also all its selector rows
    for h in range(w.heads):
        qblocks = [0, n_q - 1, (47 * h + 11) % n_q, (47 * h + 573) % n_q]
        _check_heads(w, data, keep, num, idx, o, lse, heads=[h], qblocks=qblocks,
                     budgets=np.full(w.heads, w.density), selector=h % 5 == 0 or h == w.heads - 1)
    # the fused score/select kernel on the same inputs: every row of head 5 under the gap rule
    nf, xf = fused
    assert (nf == 8 + 563).all()
    qb, kb, _ = data
    h = 5
    _say(f"[full] {w.name}: oracle selector head {h} for the fused kernel")
    _, s_ref, kk, keep_set = O.select(bf16_to_f64(qb[0, h]), bf16_to_f64(kb[0, h]), w.block, w.density, keep)
    sel = O.selectable_blocks(keep_set, w.lk, w.block)
    stats = {"exact": 0, "tolerant": 0}
    for i in range(n_q):
        stats[check_gap_rule(xf[0, h, i, : nf[0, h, i]].tolist(), s_ref[i], keep_set, sel, kk)] += 1
    _say(f"[full] {w.name}: fused head {h} rows {stats}")


def test_720p_per_head_budget_sweep_parity(gpu_lib):
    """The density sweep's per-head budgets (U[0.5, 1.5] x 10%)."""
    w = SWEEP
    budgets = head_densities(w, 0.10)
    data, keep, num, idx, o, lse = _run_full(gpu_lib, w, budgets.tolist())
    n_sel = -(-w.lk // w.block) - 8
    for h in range(w.heads):
        assert (num[0, h] == 8 + O.budget_k(float(budgets[h]), n_sel)).all()
    _check_heads(w, data, keep, num, idx, o, lse, heads=[int(np.argmax(budgets))], qblocks=[3, 1000],
                 budgets=budgets)


def test_720p_block_128_parity(gpu_lib):
    """The paper's deployed block size at the 720p shape: 72000 = 562.5 x 128,
    so the text segment [72000, 72512) straddles blocks 562 and 566 and all of
    blocks 562..566 are forced (Section 5.1's intersection rule at scale)."""
    w = P720.with_(name="720p-b128", block=128)
    data, keep, num, idx, o, lse = _run_full(gpu_lib, w, w.density)
    n_q, n_k = -(-w.lq // w.block), -(-w.lk // w.block)
    keep_set = O.keep_blocks(keep, w.lk, w.block)
    assert sorted(keep_set) == [562, 563, 564, 565, 566]
    assert (num == 5 + O.budget_k(w.density, n_k - 5)).all()
    _check_heads(w, data, keep, num, idx, o, lse, heads=[0, 11], qblocks=[0, 281, n_q - 1],
                 budgets=np.full(w.heads, w.density))


def test_pyramid_dense_scale_parity(gpu_lib):
    """The clip pyramid's first scale (2,880 queries against 75,392 keys) on the
    dense forward, as the pyramid runs it: sampled query blocks of three heads
    against the oracle's dense softmax attention."""
    import torch

    from synthetic import pyramid_scales

    w, sparse = pyramid_scales()[0]
    assert not sparse
    heads = [0, 9, 23]
    _say(f"[full] {w.name}: generating heads {heads} Lq={w.lq} Lk={w.lk}")
    qb, kb, vb = generate(w, heads=heads, workers=1)
    q, k, v = to_dev(qb), to_dev(kb), to_dev(vb)
    o, lse = gpu_lib.sparstar_dense_attn_fwd(q, k, v, w.block)
    torch.cuda.synchronize()
    o, lse = o.float().cpu().numpy(), lse.cpu().numpy()
    n_q = -(-w.lq // w.block)
    for hi, h in enumerate(heads):
        qh, kh, vh = bf16_to_f64(qb[0, hi]), bf16_to_f64(kb[0, hi]), bf16_to_f64(vb[0, hi])
        for i in (0, 17, n_q - 1):
            rows = slice(i * w.block, min((i + 1) * w.block, w.lq))
            _say(f"[full] {w.name}: oracle dense head {h} block {i}")
            o_ref, l_ref = O.dense_attention(qh[rows], kh, vh)
            check_output(o[0, hi, rows][None].astype(np.float64), o_ref[None],
                         lse[0, hi, rows][None].astype(np.float64), l_ref[None], what=f"{w.name} head {h} block {i}")


def test_pyramid_sparse_scale_parity(gpu_lib):
    """The clip pyramid's fourth scale (46,080 queries against 118,592 keys,
    fresh selection at 25%), two heads: every selector row of one head under
    the gap rule and sampled query blocks of the forward."""
    from synthetic import pyramid_scales

    w, sparse = pyramid_scales()[3]
    assert sparse
    heads = [2, 21]
    _say(f"[full] {w.name}: generating heads {heads} Lq={w.lq} Lk={w.lk}")
    qb, kb, vb = generate(w, heads=heads, workers=1)
    q, k, v = to_dev(qb), to_dev(kb), to_dev(vb)
    keep = keep_ranges(w)
    num, idx = gpu_lib.sparstar_score_blocks(q, k, w.block, w.density, keep)
    o, lse = gpu_lib.sparstar_sparse_attn_fwd(q, k, v, num, idx, w.block)
    import torch

    torch.cuda.synchronize()
    num, idx = num.cpu().numpy(), idx.cpu().numpy()
    o, lse = o.float().cpu().numpy(), lse.cpu().numpy()
    n_q, n_k = -(-w.lq // w.block), -(-w.lk // w.block)
    assert (num == 8 + O.budget_k(w.density, n_k - 8)).all()
    _check_heads(w, (qb, kb, vb), keep, num, idx, o, lse, heads=[0], qblocks=[0, 333, n_q - 1],
                 budgets=np.full(len(heads), w.density))
    _check_heads(w, (qb, kb, vb), keep, num, idx, o, lse, heads=[1], qblocks=[5, n_q - 2],
                 budgets=np.full(len(heads), w.density), selector=False)

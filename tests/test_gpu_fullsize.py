"""GPU parity at the full workload sizes, on sampled outputs the oracle can
compute one by one.

All heads run through the C ABI in the launch configuration the benchmark
times (key-range split with a workspace); the float64 oracle then recomputes
the selector of sampled heads completely (every row checked under the gap
rule) and the forward of sampled query blocks.  Coverage:
  - 720p final scale: the forward of every head on 32 stratified query blocks
    (the first and last always among them), the selector of every fifth head on
    every row, the fused selector on one head, the dense forward of every head
    on two blocks, and the clip-1 keep set (text + reference, Eq. 3's first
    branch) on every row of two heads;
  - the density sweep at 10 / 25 / 50% with per-head budgets: every budget
    count, every selector row of the largest-budget head and 8 of its blocks;
  - the mid scale, the 720p shape at the paper's 128-token blocks;
  - the clip pyramid: the dense forward of scales 1-3, the sparse scale 4 at
    25%, and the paper's scale-wise density schedule (0.625, 0.1875, 0.1875,
    0.09375 on the four finest scales) run through selector and forward on
    scales 2-5.
Inputs are generated once per session (by worker processes, before the GPU is
first used).
"""
from __future__ import annotations

import sys

import numpy as np
import pytest

import oracle as O
from synthetic import MID, P720, SWEEP, SWEEP_DENSITIES, bf16_to_f64, generate, head_densities, pyramid_scales
from tests.helpers import check_gap_rule, check_output, keep_for, to_dev

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

P720_B128 = P720.with_(name="720p-b128", block=128)
PYR_HEADS = [2, 21]          # heads of the pyramid scales that are generated
PAPER_FINEST = (0.625, 0.1875, 0.1875, 0.09375)


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="session")
def inputs():
    """Every full-size workload's bf16 inputs, generated once, before the GPU is
    initialised (so that worker processes may be used)."""
    out = {}
    for w in (P720, SWEEP, MID, P720_B128):
        _say(f"[full] generating {w.name}: H={w.heads} Lq={w.lq} Lk={w.lk}")
        out[w.name] = generate(w)
    for pw, _ in pyramid_scales():
        _say(f"[full] generating {pw.name} heads {PYR_HEADS}: Lq={pw.lq} Lk={pw.lk}")
        out[pw.name] = generate(pw, heads=PYR_HEADS)
    return out


def _stratified(n_q: int, k: int, seed: int) -> list[int]:
    """k query blocks: the first, the last, and one drawn from each of k - 2
    equal strata of the blocks in between."""
    rng = np.random.default_rng(seed)
    edges = np.linspace(1, n_q - 1, k - 1).astype(int)
    mid = [int(rng.integers(a, max(a + 1, b))) for a, b in zip(edges[:-1], edges[1:])]
    return sorted({0, n_q - 1, *mid})


def _run(lib, w, data, budget, clip=2, fused=False):
    """Selector + sparse forward on all heads, as the benchmark runs them."""
    import torch

    qb, kb, vb = data
    q, k, v = to_dev(qb), to_dev(kb), to_dev(vb)
    keep, keep_ref = keep_for(lib, w, clip)
    _say(f"[full] {w.name}: selector + sparse forward on the GPU (clip {clip})")
    num, idx = lib.sparstar_score_blocks(q, k, w.block, budget, keep)
    o, lse = lib.sparstar_sparse_attn_fwd(q, k, v, num, idx, w.block)
    extra = None
    if fused:
        _say(f"[full] {w.name}: fused score/select on the GPU")
        nf, xf = lib.sparstar_score_blocks(q, k, w.block, budget, keep, fused=True)
        extra = (nf.cpu().numpy(), xf.cpu().numpy())
    torch.cuda.synchronize()
    res = dict(keep_ref=keep_ref, num=num.cpu().numpy(), idx=idx.cpu().numpy(), o=o.float().cpu().numpy(),
               lse=lse.cpu().numpy(), fused=extra)
    del q, k, v, num, idx, o, lse
    return res


def _gpu_lists(r, h, n_q):
    return [r["idx"][0, h, i, : r["num"][0, h, i]].tolist() for i in range(n_q)]


def _check_selector(w, data, r, h, rho, lists=None):
    """Every row of head h under the gap rule; returns the row statistics."""
    qb, kb, _ = data
    n_q = -(-w.lq // w.block)
    lists = lists if lists is not None else _gpu_lists(r, h, n_q)
    _, s_ref, kk, keep_set = O.select(bf16_to_f64(qb[0, h]), bf16_to_f64(kb[0, h]), w.block, rho, r["keep_ref"])
    sel = O.selectable_blocks(keep_set, w.lk, w.block)
    stats = {"exact": 0, "tolerant": 0}
    for i in range(n_q):
        stats[check_gap_rule(lists[i], s_ref[i], keep_set, sel, kk)] += 1
    _say(f"[full] {w.name}: head {h} (rho {rho:.5f}) selector rows {stats}")
    return stats


def _check_forward(w, data, r, h, qblocks):
    """The forward of head h on the given query blocks, on the GPU's own lists."""
    qb, kb, vb = data
    n_q = -(-w.lq // w.block)
    lists = _gpu_lists(r, h, n_q)
    qh, kh, vh = bf16_to_f64(qb[0, h]), bf16_to_f64(kb[0, h]), bf16_to_f64(vb[0, h])
    for i in qblocks:
        rows = slice(i * w.block, min((i + 1) * w.block, w.lq))
        o_ref, l_ref = O.sparse_attention(qh[rows], kh, vh, [lists[i]], w.block)
        check_output(r["o"][0, h, rows][None].astype(np.float64), o_ref[None],
                     r["lse"][0, h, rows][None].astype(np.float64), l_ref[None], what=f"{w.name} head {h} block {i}")


def test_720p_final_scale_parity(gpu_lib, inputs):
    w = P720
    data = inputs[w.name]
    r = _run(gpu_lib, w, data, w.density, fused=True)
    n_q = -(-w.lq // w.block)
    assert (r["num"] == 8 + 563).all()
    for h in range(w.heads):
        qblocks = _stratified(n_q, 32, seed=1000 + h)
        assert len(qblocks) == 32 and qblocks[0] == 0 and qblocks[-1] == n_q - 1
        _say(f"[full] {w.name}: forward of head {h} on 32 stratified query blocks")
        _check_forward(w, data, r, h, qblocks)
        if h % 5 == 0 or h == w.heads - 1:
            _check_selector(w, data, r, h, w.density)
    # the fused score/select kernel on the same inputs: every row of head 5
    nf, xf = r["fused"]
    assert (nf == 8 + 563).all()
    _check_selector(w, data, r, 5, w.density, lists=[xf[0, 5, i, : nf[0, 5, i]].tolist() for i in range(n_q)])


def test_720p_dense_parity(gpu_lib, inputs):
    """The in-house dense forward at 720p (the denominator of every sparse/dense
    speedup): every head on two query blocks against the oracle's dense softmax
    attention over all 144,512 keys."""
    import torch

    w = P720
    qb, kb, vb = inputs[w.name]
    _say(f"[full] {w.name}: dense forward on the GPU")
    o, lse = gpu_lib.sparstar_dense_attn_fwd(to_dev(qb), to_dev(kb), to_dev(vb), w.block)
    torch.cuda.synchronize()
    o, lse = o.float().cpu().numpy(), lse.cpu().numpy()
    n_q = -(-w.lq // w.block)
    for h in range(w.heads):
        qh, kh, vh = bf16_to_f64(qb[0, h]), bf16_to_f64(kb[0, h]), bf16_to_f64(vb[0, h])
        for i in (0 if h % 2 == 0 else n_q - 1, (97 * h + 31) % n_q):
            rows = slice(i * w.block, min((i + 1) * w.block, w.lq))
            o_ref, l_ref = O.dense_attention(qh[rows], kh, vh)
            check_output(o[0, h, rows][None].astype(np.float64), o_ref[None], lse[0, h, rows][None].astype(np.float64),
                         l_ref[None], what=f"{w.name} dense head {h} block {i}")
    _say(f"[full] {w.name}: dense forward checked on {2 * w.heads} blocks")


def test_720p_clip1_parity(gpu_lib, inputs):
    """Eq. 3's first branch at 720p: clip 1 keeps the text and the reference
    dense (1,133 forced blocks), so only the 1,125 current-scale blocks are
    ranked and k = ceil(0.25 x 1125) = 282."""
    w = P720
    data = inputs[w.name]
    r = _run(gpu_lib, w, data, w.density, clip=1)
    keep_set = O.keep_blocks(r["keep_ref"], w.lk, w.block)
    assert len(keep_set) == 1133
    assert (r["num"] == 1133 + O.budget_k(w.density, 1125)).all() and O.budget_k(w.density, 1125) == 282
    n_q = -(-w.lq // w.block)
    for h in (3, 17):
        _check_selector(w, data, r, h, w.density)
        _check_forward(w, data, r, h, _stratified(n_q, 6, seed=77 + h))


@pytest.mark.parametrize("rho", SWEEP_DENSITIES)
def test_720p_sweep_parity(gpu_lib, inputs, rho):
    """The density sweep with per-head budgets U[0.5, 1.5] x rho: every head's
    count, every selector row of the largest-budget head and 8 of its blocks."""
    w = SWEEP
    data = inputs[w.name]
    budgets = head_densities(w, rho)
    r = _run(gpu_lib, w, data, budgets.tolist())
    n_sel = -(-w.lk // w.block) - 8
    for h in range(w.heads):
        assert (r["num"][0, h] == 8 + O.budget_k(float(budgets[h]), n_sel)).all()
    h = int(np.argmax(budgets))
    _check_selector(w, data, r, h, float(budgets[h]))
    _check_forward(w, data, r, h, _stratified(-(-w.lq // w.block), 8, seed=int(rho * 1000)))


def test_mid_scale_parity(gpu_lib, inputs):
    w = MID
    data = inputs[w.name]
    r = _run(gpu_lib, w, data, w.density)
    n_q = -(-w.lq // w.block)
    for h in (0, 13, 23):
        _check_selector(w, data, r, h, w.density)
        _check_forward(w, data, r, h, [0, 1, 90, n_q - 1])


def test_720p_block_128_parity(gpu_lib, inputs):
    """The paper's deployed block size at the 720p shape: 72000 = 562.5 x 128,
    so the text segment [72000, 72512) straddles blocks 562 and 566 and all of
    blocks 562..566 are forced (Section 5.1's intersection rule at scale)."""
    w = P720_B128
    data = inputs[w.name]
    r = _run(gpu_lib, w, data, w.density)
    n_q, n_k = -(-w.lq // w.block), -(-w.lk // w.block)
    keep_set = O.keep_blocks(r["keep_ref"], w.lk, w.block)
    assert sorted(keep_set) == [562, 563, 564, 565, 566]
    assert (r["num"] == 5 + O.budget_k(w.density, n_k - 5)).all()
    for h in (0, 11):
        _check_selector(w, data, r, h, w.density)
        _check_forward(w, data, r, h, [0, 281, n_q - 1])


@pytest.mark.parametrize("scale", [1, 2, 3])
def test_pyramid_dense_scale_parity(gpu_lib, inputs, scale):
    """The clip pyramid's dense scales 1-3 (2,880 / 11,520 / 25,920 queries
    against 72,512 + Lq keys), as the pyramid runs them: sampled query blocks
    of the generated heads against the oracle's dense softmax attention."""
    import torch

    w, sparse = pyramid_scales()[scale - 1]
    assert not sparse
    qb, kb, vb = inputs[w.name]
    o, lse = gpu_lib.sparstar_dense_attn_fwd(to_dev(qb), to_dev(kb), to_dev(vb), w.block)
    torch.cuda.synchronize()
    o, lse = o.float().cpu().numpy(), lse.cpu().numpy()
    n_q = -(-w.lq // w.block)
    for hi, h in enumerate(PYR_HEADS):
        qh, kh, vh = bf16_to_f64(qb[0, hi]), bf16_to_f64(kb[0, hi]), bf16_to_f64(vb[0, hi])
        for i in (0, (37 * h + 17) % n_q, n_q - 1):
            rows = slice(i * w.block, min((i + 1) * w.block, w.lq))
            o_ref, l_ref = O.dense_attention(qh[rows], kh, vh)
            check_output(o[0, hi, rows][None].astype(np.float64), o_ref[None],
                         lse[0, hi, rows][None].astype(np.float64), l_ref[None], what=f"{w.name} head {h} block {i}")
    _say(f"[full] {w.name}: dense forward checked")


def test_pyramid_sparse_scale_parity(gpu_lib, inputs):
    """The clip pyramid's fourth scale (46,080 queries against 118,592 keys,
    fresh selection at 25%): every selector row of one head under the gap rule
    and sampled query blocks of the forward of both generated heads."""
    w, sparse = pyramid_scales()[3]
    assert sparse
    data = inputs[w.name]
    r = _run(gpu_lib, w, data, w.density)
    n_q, n_k = -(-w.lq // w.block), -(-w.lk // w.block)
    assert (r["num"] == 8 + O.budget_k(w.density, n_k - 8)).all()
    _check_selector(w, data, r, 0, w.density)
    _check_forward(w, data, r, 0, [0, 333, n_q - 1])
    _check_forward(w, data, r, 1, [5, n_q - 2])


def test_pyramid_paper_density_schedule_parity(gpu_lib, inputs):
    """Section 5.2's scale-wise density schedule through the kernels: the
    paper's 720p densities of the four finest scales (0.625, 0.1875, 0.1875,
    0.09375; supplement, sparsity schedule) assigned by query length to the
    pyramid (sparstar_scale_densities, checked against the oracle's schedule),
    then selector and forward on every sparsified scale (2-5) with its own
    budget: every selector row of one head under the gap rule, and sampled
    query blocks of both generated heads."""
    scales = pyramid_scales()
    lqs = [pw.lq for pw, _ in scales]
    rho = gpu_lib.sparstar_scale_densities(lqs, PAPER_FINEST)
    assert rho == O.scale_densities(lqs, list(PAPER_FINEST))
    assert rho[0] is None and rho[1:] == list(PAPER_FINEST)
    for (pw, _), r_s in zip(scales[1:], rho[1:]):
        w = pw.with_(density=r_s)
        data = inputs[pw.name]
        r = _run(gpu_lib, w, data, r_s)
        n_q, n_k = -(-w.lq // w.block), -(-w.lk // w.block)
        assert (r["num"] == 8 + O.budget_k(r_s, n_k - 8)).all()
        _check_selector(w, data, r, 1, r_s)
        _check_forward(w, data, r, 0, _stratified(n_q, 4, seed=w.lq))
        _check_forward(w, data, r, 1, _stratified(n_q, 4, seed=w.lq + 1))

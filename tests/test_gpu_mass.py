"""GPU parity of the retained-attention-mass diagnostic (Section 4 analysis)
against the float64 oracle, through the C ABI.

Tolerances
  - sparstar_retained_mass on given fp32 log-sum-exps: relative 1e-6 (one fp32
    subtraction and expf).
  - retained mass from the kernels' own sparse and dense lse: each lse is within
    LSE_ABS of the exact value, so exp(lse_sel - lse_all) is within a relative
    exp(2 LSE_ABS) - 1 of the exact mass.
  - sparstar_token_topk_mass with the exact (oracle) lse: each logit is an fp32
    dot product of bf16 inputs (exact products, D rounded additions: error at
    most D u s sum_d |q_d k_d|, u = 2^-24), then one subtraction of the fp32
    lse (2 u (1 + |lse|)); the weights are summed in fp32 per lane over Lk/256
    terms and then over a 256-wide tree ((Lk/256 + 8) u relative).  A swap of
    two logits closer than the logit error at the n-th place stays inside the
    same bound.
  - with the dense kernel's lse: a relative exp(LSE_ABS) - 1 on top of that.
"""
from __future__ import annotations

import math
import sys

import numpy as np
import pytest

import oracle as O
from synthetic import P720, TINY, bf16_to_f64, generate
from tests.helpers import keep_for, LSE_ABS, lists_from_device, to_dev

pytestmark = pytest.mark.gpu

MASS_REL_E2E = math.exp(2 * LSE_ABS) - 1
U32 = 2.0 ** -24


def _topk_tol(qr, kh, scale, lse_rows, ref):
    """A-priori bound on |GPU - oracle| of the token top-n mass (module docstring)."""
    d = qr.shape[1]
    s = scale if scale else 1.0 / math.sqrt(d)
    logit = 1.01 * d * U32 * s * (np.abs(qr) @ np.abs(kh).T).max(axis=1) + 2 * U32 * (1 + np.abs(lse_rows))
    summ = (kh.shape[0] / 256 + 8) * U32
    return ref * (np.expm1(logit) + summ + 4 * U32) + 1e-7


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _lse64(q, k, scale=None):
    """Dense log-sum-exp in float64 (the oracle's dense attention)."""
    v = np.zeros_like(k[:, :1])
    _, lse = O.dense_attention(q, k, v, scale)
    return lse


def test_retained_mass_formula(gpu_lib):
    import torch

    _say("[mass] elementwise exp(lse_sel - lse_all)")
    rng = np.random.default_rng(1)
    n = 70_001  # several grid strides' worth plus a ragged tail
    lse_all = rng.uniform(-5, 20, n).astype(np.float32)
    lse_sel = (lse_all - np.abs(rng.standard_normal(n)) * 3).astype(np.float32)
    lse_sel[::97] = -np.inf
    lse_sel[5] = lse_all[5]
    sel_d, all_d = torch.from_numpy(lse_sel).cuda(), torch.from_numpy(lse_all).cuda()
    got = gpu_lib.sparstar_retained_mass(sel_d, all_d).cpu().numpy().astype(np.float64)
    d = lse_sel.astype(np.float64) - lse_all.astype(np.float64)
    ref = np.where(np.isneginf(lse_sel), 0.0, np.exp(d))
    np.testing.assert_allclose(got, ref, rtol=1e-6, atol=0)
    assert got[5] == 1.0 and (got[::97] == 0).all()
    # in place over lse_sel
    gpu_lib.sparstar_retained_mass(sel_d, all_d, out=sel_d)
    np.testing.assert_allclose(sel_d.cpu().numpy().astype(np.float64), ref, rtol=1e-6, atol=0)


def _tiny_inputs(w=TINY):
    qb, kb, vb = generate(w)
    return (qb, kb, vb), (to_dev(qb), to_dev(kb), to_dev(vb))


def test_retained_mass_end_to_end_tiny(gpu_lib):
    import torch

    w = TINY
    _say(f"[mass] end to end {w.name}: selector, sparse and dense forward, mass")
    (qb, kb, vb), (q, k, v) = _tiny_inputs(w)
    keep, _ = keep_for(gpu_lib, w)
    num, idx = gpu_lib.sparstar_score_blocks(q, k, w.block, w.density, keep)
    _, lse_sel = gpu_lib.sparstar_sparse_attn_fwd(q, k, v, num, idx, w.block)
    _, lse_all = gpu_lib.sparstar_dense_attn_fwd(q, k, v, w.block)
    mass = gpu_lib.sparstar_retained_mass(lse_sel, lse_all)
    torch.cuda.synchronize()
    lists = lists_from_device(num, idx)[0]
    m = mass.cpu().numpy().astype(np.float64)
    for h in range(w.heads):
        qh, kh = bf16_to_f64(qb[0, h]), bf16_to_f64(kb[0, h])
        ref = O.retained_mass(qh, kh, lists[h], w.block)
        err = np.abs(m[0, h] - ref)
        assert (err <= MASS_REL_E2E * ref + 1e-6).all(), f"head {h}: max |dmass| {err.max():.3e}"
        assert (m[0, h] > 0).all() and (m[0, h] <= 1 + MASS_REL_E2E).all()


def _topk_case(gpu_lib, qb, kb, rows, n_tok, scale=None, lse_all=None):
    """Run the token top-n kernel on every head of (qb, kb) and compare it with
    the oracle on the sampled rows.  n_tok: [H, n_rows] int."""
    import torch

    _, H, Lq, D = qb.shape
    q, k = to_dev(qb), to_dev(kb)
    lse_ref = [_lse64(bf16_to_f64(qb[0, h]), bf16_to_f64(kb[0, h]), scale) for h in range(H)]
    if lse_all is None:
        lse_all = torch.from_numpy(np.stack(lse_ref)[None].astype(np.float32)).cuda()
    nt = torch.from_numpy(np.asarray(n_tok, dtype=np.int32)[None].copy()).cuda()
    got = gpu_lib.sparstar_token_topk_mass(q, k, rows, nt, lse_all, scale or 0.0).cpu().numpy().astype(np.float64)
    for h in range(H):
        qh, kh = bf16_to_f64(qb[0, h]), bf16_to_f64(kb[0, h])
        ref = O.token_topk_mass(qh[rows], kh, np.asarray(n_tok[h]), scale)
        err = np.abs(got[0, h] - ref)
        tol = _topk_tol(qh[rows], kh, scale, lse_ref[h][rows], ref)
        assert (err <= tol).all(), f"head {h}: |dmass| {err.max():.3e}, worst err/tol {(err / tol).max():.2f}"
    return got[0]


def test_token_topk_mass_edge_counts(gpu_lib):
    w = TINY
    _say(f"[mass] token top-n {w.name}: counts 0, 1, Lk, beyond Lk, negative")
    (qb, kb, _), _ = _tiny_inputs(w)
    lk = kb.shape[2]
    rows = [0, 1, 63, 64, 200, 511]
    n_tok = [[0, 1, 17, lk, lk + 5, -3], [lk // 4, 1000, 2, lk - 1, 64, 511]]
    got = _topk_case(gpu_lib, qb, kb, rows, n_tok)
    assert got[0, 0] == 0.0 and got[0, 5] == 0.0
    assert abs(got[0, 3] - 1.0) <= 1e-4 and got[0, 4] == got[0, 3]


def test_token_topk_mass_exact_ties(gpu_lib):
    """Repeated key rows give logits that are equal in fp32 as well; counts that
    end inside a group of equal logits take part of the group."""
    _say("[mass] token top-n with tied logits")
    rng = np.random.default_rng(9)
    H, Lq, Lk, D = 2, 64, 1500, 64
    from synthetic.workloads import bf16_bits

    q = bf16_bits(rng.standard_normal((1, H, Lq, D)).astype(np.float32))
    base = rng.standard_normal((1, H, 100, D)).astype(np.float32) * 1.5
    k = bf16_bits(np.repeat(base, 15, axis=2))  # each key row 15 times
    rows = [0, 7, 63]
    n_tok = [[1, 15, 22], [30, 37, 1499]]
    _topk_case(gpu_lib, q, k, rows, n_tok)


@pytest.mark.parametrize("sharp", [False, True], ids=["tau", "4tau"])
def test_token_topk_mass_d128_ragged(gpu_lib, sharp):
    _say(f"[mass] token top-n D=128, ragged Lk, sharp={sharp}")
    rng = np.random.default_rng(17)
    H, Lq, Lk, D = 3, 130, 2500, 128
    from synthetic.workloads import bf16_bits

    q = bf16_bits(rng.standard_normal((1, H, Lq, D)).astype(np.float32))
    k = bf16_bits(rng.standard_normal((1, H, Lk, D)).astype(np.float32))
    scale = 4 / math.sqrt(D) if sharp else None
    rows = list(range(0, Lq, 9))  # 15 rows
    n_tok = rng.integers(0, Lk + 1, size=(H, len(rows)))
    _topk_case(gpu_lib, q, k, rows, n_tok, scale)


def test_mass_at_720p_sampled(gpu_lib):
    """The 720p final scale (72,000 queries, 144,512 keys, D = 128, b = 64,
    rho = 0.25), two heads: the block selection's retained mass from the two
    kernels' lse on every query, checked against the oracle on sampled query
    blocks, and the token bound with the dense kernel's lse on sampled rows,
    with n = the real keys of A_i."""
    import torch

    w = P720
    heads = [0, 17]
    _say(f"[mass] {w.name}: generating heads {heads}")
    qb, kb, vb = generate(w, heads=heads, workers=1)
    q, k, v = to_dev(qb), to_dev(kb), to_dev(vb)
    keep, _ = keep_for(gpu_lib, w)
    _say(f"[mass] {w.name}: selector, sparse and dense forward")
    num, idx = gpu_lib.sparstar_score_blocks(q, k, w.block, w.density, keep)
    _, lse_sel = gpu_lib.sparstar_sparse_attn_fwd(q, k, v, num, idx, w.block)
    _, lse_all = gpu_lib.sparstar_dense_attn_fwd(q, k, v, w.block)
    mass = gpu_lib.sparstar_retained_mass(lse_sel, lse_all)
    lists = lists_from_device(num, idx)[0]
    lk, b = w.lk, w.block
    rows = [0, 63, 35_000, 71_999]
    n_tok = np.array([[sum(min((j + 1) * b, lk) - j * b for j in lists[h][r // b]) for r in rows]
                      for h in range(len(heads))])
    nt = torch.from_numpy(n_tok.astype(np.int32)[None].copy()).cuda()
    bound = gpu_lib.sparstar_token_topk_mass(q, k, rows, nt, lse_all)
    torch.cuda.synchronize()
    m = mass.cpu().numpy().astype(np.float64)[0]
    bd = bound.cpu().numpy().astype(np.float64)[0]
    n_q = -(-w.lq // b)
    for hi in range(len(heads)):
        qh, kh = bf16_to_f64(qb[0, hi]), bf16_to_f64(kb[0, hi])
        for i in (0, 547, n_q - 1):
            t = slice(i * b, min((i + 1) * b, w.lq))
            _say(f"[mass] {w.name}: oracle head {heads[hi]} block {i}")
            ref = O.retained_mass(qh[t], kh, [lists[hi][i]], b)
            err = np.abs(m[hi, t] - ref)
            assert (err <= MASS_REL_E2E * ref + 1e-6).all(), f"head {heads[hi]} block {i}: {err.max():.3e}"
        ref_b = O.token_topk_mass(qh[rows], kh, n_tok[hi])
        lse_rows = _lse64(qh[rows], kh)
        tol = _topk_tol(qh[rows], kh, None, lse_rows, ref_b) + math.expm1(LSE_ABS) * ref_b
        err = np.abs(bd[hi] - ref_b)
        assert (err <= tol).all(), f"head {heads[hi]}: |dmass| {err.max():.3e}"
        # the block selection never beats the best equally many single keys
        assert (m[hi, rows] <= bd[hi] * (1 + MASS_REL_E2E) + 1e-6).all()

"""Test-side helpers: tensor marshalling, the selection gap rule, list checks.

Nothing here computes the method; the oracle does that."""
from __future__ import annotations

import numpy as np

GAP = 1e-3          # selection: exact match required where the boundary gap exceeds this
O_MAX_ABS = 1e-2    # output: max |dO| (bf16 inputs, fp32-accumulated reference)
O_REL_FRO = 1e-2    # output: per-head relative Frobenius error
# log-sum-exp: max |dlse| (the bound the parity rules set).  The kernel takes lse
# from an fp32 sum of the unrounded softmax numerators, so only fp32 rounding of
# the logits, the exponentials and the sums separates it from the float64
# value (about 1e-5 at these sizes).
LSE_ABS = 1e-3


def keep_for(lib, w, clip: int = 2):
    """Eq. 3's forced token ranges for the workload's text and reference
    segments: (the library's, sparstar_clip_keep_ranges, for the GPU calls; the
    oracle's, keep_ranges_for_clip, for the oracle calls).  They must agree."""
    import oracle as O

    seg = w.segments()
    k_lib = lib.sparstar_clip_keep_ranges(clip, seg["text"], seg["ref"])
    k_ref = O.keep_ranges_for_clip(clip, seg["text"], seg["ref"])
    assert [tuple(r) for r in k_lib] == [tuple(r) for r in k_ref], (k_lib, k_ref)
    return k_lib, k_ref


def to_dev(bits: np.ndarray):
    """bf16 bit patterns (uint16) -> a contiguous bf16 tensor on the GPU."""
    import torch

    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def bf16_tensor_to_f64(t) -> np.ndarray:
    import torch

    return t.detach().to(torch.float32).cpu().numpy().astype(np.float64)


def lists_from_device(num, idx) -> list:
    """[B,H,n_q] counts + [B,H,n_q,stride] indices -> nested python lists."""
    n = num.cpu().numpy()
    ix = idx.cpu().numpy()
    out = []
    for b in range(n.shape[0]):
        out.append([[ix[b, h, i, : n[b, h, i]].tolist() for i in range(n.shape[2])] for h in range(n.shape[1])])
    return out


def lists_to_device(lists_bh, n_q: int, stride: int | None = None):
    """Nested [B][H][n_q] lists -> (num, idx) int32 tensors on the GPU."""
    import torch

    B, H = len(lists_bh), len(lists_bh[0])
    stride = stride or max(1, max(len(l) for bl in lists_bh for hl in bl for l in hl))
    num = np.zeros((B, H, n_q), np.int32)
    idx = np.full((B, H, n_q, stride), -7, np.int32)
    for b in range(B):
        for h in range(H):
            for i, l in enumerate(lists_bh[b][h]):
                num[b, h, i] = len(l)
                idx[b, h, i, : len(l)] = l
    return torch.from_numpy(num).cuda(), torch.from_numpy(idx).cuda()


def check_gap_rule(gpu_list, oracle_row_scores, keep, sel, k):
    """Compare one GPU row with the oracle's float64 scores under the gap rule.

    Returns "exact" or "tolerant"; raises AssertionError on a violation."""
    keep_set = set(keep)
    assert gpu_list == sorted(set(gpu_list)), "list not strictly ascending"
    assert keep_set <= set(gpu_list), "a forced block is missing"
    chosen = [j for j in gpu_list if j not in keep_set]
    assert len(chosen) == k, f"selected {len(chosen)} blocks, budget {k}"
    assert all(j in set(sel) for j in chosen)
    if k == 0:
        return "exact"
    s = oracle_row_scores
    order = sorted(sel, key=lambda j: (-s[j], j))
    ref = set(order[:k])
    t_k = s[order[k - 1]]
    t_k1 = s[order[k]] if k < len(order) else -np.inf
    if t_k - t_k1 > GAP:
        assert set(chosen) == ref, "selection differs where the boundary gap exceeds 1e-3"
        return "exact"
    must = {j for j in sel if s[j] > t_k + GAP}
    never = {j for j in sel if s[j] < t_k1 - GAP}
    assert must <= set(chosen), "a clearly-above-threshold block was dropped"
    assert not (never & set(chosen)), "a clearly-below-threshold block was taken"
    return "tolerant"


# Sharpened-softmax stress cases (scale 4 / sqrt(D)): few keys dominate, so the
# bf16 rounding of P (relative 2^-9) shows directly, |dO| <= 2^-9 max|v| + the
# bf16 rounding of O (2^-9 |O|); with |v|, |O| <= 4 that is <= 1.6e-2.
O_MAX_ABS_SHARP = 1.6e-2
LSE_ABS_SHARP = LSE_ABS


def check_output(o_gpu: np.ndarray, o_ref: np.ndarray, lse_gpu=None, lse_ref=None, what="", max_abs=O_MAX_ABS,
                 lse_abs=LSE_ABS):
    """O: max-abs and per-head relative Frobenius; lse: max-abs.  Arrays [.., L, D]."""
    d = np.abs(o_gpu - o_ref)
    assert d.max() <= max_abs, f"{what}: max |dO| = {d.max():.3e}"
    num = np.sqrt(((o_gpu - o_ref) ** 2).sum(axis=(-2, -1)))
    den = np.sqrt((o_ref ** 2).sum(axis=(-2, -1)))
    rel = num / np.maximum(den, 1e-30)
    assert rel.max() <= O_REL_FRO, f"{what}: relative Frobenius error {rel.max():.3e}"
    if lse_gpu is not None:
        fin = np.isfinite(lse_ref)
        assert (np.isfinite(lse_gpu) == fin).all(), f"{what}: lse finiteness differs"
        if fin.any():
            dl = np.abs(lse_gpu[fin] - lse_ref[fin]).max()
            assert dl <= lse_abs, f"{what}: max |dlse| = {dl:.3e}"
    return float(d.max())

"""GPU parity of sparstar_score_blocks_static (the selector with its scratch in
the library's static per-GPU buffer) against sparstar_score_blocks, through the
C ABI: two calls in a row, the second with a smaller input, each bit-exact
against the workspace entry point (the same kernels on the same inputs), with
the scratch still holding the previous call's contents."""
from __future__ import annotations

import sys

import numpy as np
import pytest

from synthetic import TINY, generate
from tests.helpers import to_dev

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _keep(lib, w):
    seg = w.segments()
    return lib.sparstar_clip_keep_ranges(2, seg["text"], seg["ref"])


def _pair(lib, w, budget, with_scores):
    """(workspace entry point, static entry point) outputs on the same inputs."""
    import torch

    qb, kb, _ = generate(w)
    q, k = to_dev(qb), to_dev(kb)
    keep = _keep(lib, w)
    B, H, Lq, D = q.shape
    Lk = k.shape[2]
    n_q, n_k = -(-Lq // w.block), -(-Lk // w.block)
    stride = lib.sparstar_kv_stride(H, Lk, w.block, budget, keep)
    s_ref = torch.full((B, H, n_q, n_k), float("nan"), device="cuda") if with_scores else None
    s_sta = torch.full((B, H, n_q, n_k), float("nan"), device="cuda") if with_scores else None
    num_r, idx_r = lib.sparstar_score_blocks(q, k, w.block, budget, keep, kv_stride=stride, scores=s_ref)
    # preallocated outputs, poisoned, so that nothing is allocated around the static call
    num_s = torch.full_like(num_r, -9)
    idx_s = torch.full_like(idx_r, -9)
    torch.cuda.synchronize()
    lib.sparstar_score_blocks_static(q, k, w.block, budget, keep, kv_stride=stride, scores=s_sta,
                                     out=(num_s, idx_s))
    torch.cuda.synchronize()
    return (num_r, idx_r, s_ref), (num_s, idx_s, s_sta)


def _check(ref, got, what):
    num_r, idx_r, s_r = ref
    num_s, idx_s, s_s = got
    n = num_r.cpu().numpy()
    assert np.array_equal(n, num_s.cpu().numpy()), f"{what}: counts differ"
    ir, is_ = idx_r.cpu().numpy(), idx_s.cpu().numpy()
    for b in range(n.shape[0]):
        for h in range(n.shape[1]):
            for i in range(n.shape[2]):
                c = n[b, h, i]
                assert np.array_equal(ir[b, h, i, :c], is_[b, h, i, :c]), f"{what}: list ({b},{h},{i}) differs"
    if s_r is not None:
        # forced columns are unspecified; every selectable score must agree bit for bit
        a, c = s_r.cpu().numpy(), s_s.cpu().numpy()
        fin = ~np.isnan(a)
        assert np.array_equal(a[fin], c[fin]), f"{what}: scores differ"


def test_static_scratch_selector_matches_workspace_selector(gpu_lib):
    lib = gpu_lib
    # call 1: 8 heads, D 128, ragged lengths, S inside the static scratch
    w1 = TINY.with_(name="static1", heads=8, head_dim=128, lq=64 * 100 + 13, l_ref=64 * 700 + 21, l_text=512,
                    seed=61, aligned=6, density=0.3)
    budgets = [0.1 + 0.05 * h for h in range(w1.heads)]
    _say(f"[static] call 1: H={w1.heads} D={w1.head_dim} Lq={w1.lq} Lk={w1.lk}, S in the scratch")
    ref, got = _pair(lib, w1, budgets, with_scores=False)
    _check(ref, got, "call 1")
    # call 2: a smaller input (2 heads, D 64), S written to the caller's buffer;
    # the scratch still holds call 1's pooled blocks and scores
    w2 = TINY.with_(name="static2", seed=62)
    _say(f"[static] call 2: H={w2.heads} D={w2.head_dim} Lq={w2.lq} Lk={w2.lk}, S in the caller's buffer")
    ref, got = _pair(lib, w2, w2.density, with_scores=True)
    _check(ref, got, "call 2")
    # call 3: the first shape again, now with S outside the scratch
    _say("[static] call 3: call 1's shape with S in the caller's buffer")
    ref, got = _pair(lib, w1, budgets, with_scores=True)
    _check(ref, got, "call 3")


def test_static_scratch_rejects_what_does_not_fit(gpu_lib):
    """Sizes whose scratch exceeds the static buffer fail on the host with
    SPARSTAR_ERR_WORKSPACE, and the outputs stay untouched."""
    import torch

    lib = gpu_lib
    H, Lq, Lk, D, b = 24, 72_000, 144_512, 128, 64
    q = torch.zeros((1, H, Lq, D), dtype=torch.bfloat16, device="cuda")
    k = torch.zeros((1, H, Lk, D), dtype=torch.bfloat16, device="cuda")
    keep = [(72_000, 72_512)]
    num = torch.full((1, H, Lq // b), -9, dtype=torch.int32, device="cuda")
    idx = torch.full((1, H, Lq // b, 571), -9, dtype=torch.int32, device="cuda")
    with pytest.raises(lib.SparstarError) as e:
        lib.sparstar_score_blocks_static(q, k, b, 0.25, keep, out=(num, idx))
    assert e.value.code == lib.ERR_WORKSPACE and "67108864" in str(e.value)
    torch.cuda.synchronize()
    assert (num == -9).all() and (idx == -9).all()

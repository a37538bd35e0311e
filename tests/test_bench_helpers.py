"""Host-side helpers of bench.py: the executed-FLOP count it reports."""
from __future__ import annotations

import numpy as np

import bench


def _brute(lists, lq, lk, block, d):
    total = 0
    for i, row in enumerate(lists):
        rows = min(block, lq - i * block)
        keys = sum(min(block, lk - j * block) for j in row)
        total += 4 * rows * keys * d
    return float(total)


def test_executed_flops_counts_real_rows_and_keys():
    rng = np.random.default_rng(3)
    for lq, lk, block, d in [(512, 1152, 64, 64), (700, 1300, 128, 128), (72_000, 144_512, 128, 128),
                             (130, 70, 64, 32)]:
        n_q, n_k = -(-lq // block), -(-lk // block)
        lists = [sorted(rng.choice(n_k, size=rng.integers(0, n_k + 1), replace=False).tolist()) for _ in range(n_q)]
        stride = n_k
        num = np.array([[len(r) for r in lists]], dtype=np.int32)
        idx = np.zeros((1, n_q, stride), dtype=np.int32)
        for i, r in enumerate(lists):
            idx[0, i, : len(r)] = r
        last = np.take_along_axis(idx, np.clip(num - 1, 0, None)[..., None].astype(np.int64), axis=-1)[..., 0]
        got = bench.executed_flops(num, last, lq, lk, block, d)
        assert got == _brute(lists, lq, lk, block, d)
